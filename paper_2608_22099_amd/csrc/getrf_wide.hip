// Wide-band LU with partial pivoting in one persistent launch: the case of
// Sec. III-A's specialised algorithm f(N) where kl is large enough that each
// panel's trailing update is a real dense product (xGBTRF semantics for the
// factors, ipiv and info).
//
// The band is cut into blocks of NB = 32 columns.  Panel k (columns 32k ..
// 32k+31) reaches the nblk = (kl+ku+31)/32 blocks to its right, so
// G = nblk + 1 workgroups keep every block that is still being updated
// resident: workgroup w owns blocks w, w+G, w+2G, ...  A block lives in LDS
// as a window of 288 = NB + 256 band rows: the rows the panel being applied
// reaches.  For each panel k before it the owner
//   1. waits until panel k is published (a device-scope counter, bounded wait),
//   2. applies its row interchanges (one gather by the panel's net permutation),
//   3. forms U12 = L11^-1 * (top 32 rows) by forward substitution,
//   4. updates the rows below, A22 += (-L21) * U12, with v_mfma_f64_16x16x4f64,
//   5. writes the top 32 rows back (they are final) and loads the 32 band rows
//      that enter the window at the bottom.
// When all panels before it are applied the block is itself the next panel:
// its owner factors it in place (first with every pivot on the diagonal,
// verified column by column against partial pivoting; on the first failure
// again with partial pivoting), publishes the panel's L (in the row order
// after the panel's interchanges, laid out for the matrix-core operands) in a
// ring of G slots, and then writes the factors to the band (nothing on the
// chain reads them there).  The owner of the next block applies the panel at
// once, so the chain of panels never waits for a relaunch, and the band is
// read from HBM once and written once.
//
// Every update of an entry is one fused multiply-add in the order of the
// column steps (forward substitution and the matrix-core product both sum in
// that order), with the multipliers formed as in the unblocked algorithm.
// Beyond each step's update extent the blocked form also updates entries
// that are structural zeros, which can change the sign of a zero and carry a
// NaN multiplier into them; on finite data the factors are those of the
// unblocked algorithm.
#include <algorithm>
#include <cfloat>
#include <climits>
#include <cstdlib>
#include <utility>

#include "common.hpp"
#include "wave.hpp"

namespace bandlu {

int launch_getrf_wide(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s, void *scratch, size_t scratch_bytes,
                      double *dB, int64_t ldb, int64_t strideB, int64_t nrhs);
bool getrf_wide_fits(int64_t n, int64_t kl, int64_t ku, int64_t batch);
bool getrf_wide_fused_fits(int64_t n, int64_t kl, int64_t ku, int64_t nrhs);
bool getrf_wide_one_launch(int64_t n, int64_t kl, int64_t ku, int64_t batch);
size_t getrf_wide_scratch_bytes(int64_t n, int64_t kl, int64_t ku, int64_t batch);

namespace {

typedef double v4d __attribute__((ext_vector_type(4)));

constexpr int NB = 32;               // panel width = block width
constexpr int kMaxKl = 256;
constexpr int PR = NB + kMaxKl;      // rows of a block window
constexpr int LDW = NB + 1;          // row stride of a window in LDS (doubles)
constexpr int kThreads = 320;        // wave 0: rows 0..31; waves 1..4: rows 32..287
constexpr int kWaves = kThreads / 64;
constexpr int LDU = NB + 2;          // published pivot rows: value c at [s * LDU + c], 1/pivot at NB
constexpr int kHdrBytes = 256;       // per matrix: {panels published, failed}
// slot of a published panel: int perm[288], int ident, padding to 1280 bytes,
// then L11 (32 x 32, column-major, unit lower, only r > s used) and -L21
// (256 x 32, column-major), written by the rows that hold them with
// consecutive rows at consecutive addresses
constexpr int kSlotInts = 320;
constexpr size_t kSlotBytes = size_t(kSlotInts) * 4 + size_t(NB) * NB * 8 + size_t(PR - NB) * NB * 8;

struct WideParams {
    double *AB;
    int32_t *ipiv;
    int32_t *info;
    char *scratch;
    int64_t ldab, strideAB, strideP, scratch_stride;
    int n, kl, ku, nblk, G, nblocks;
    int b0;          // first matrix of this launch
    unsigned spin_limit;
    // right-hand sides for the fused forward substitution (null: none); the
    // workgroup after the G block owners applies each panel to them
    double *B;
    int64_t ldb, strideB;
    int nrhs;
};

__device__ __forceinline__ int prow(int r) { return r % PR; }

// A value the optimiser may not see through: addresses built from it are
// formed where they are used instead of being hoisted out of the block and
// panel loops and kept live (32 column or row offsets at a time would not fit
// the registers).
template <typename T>
__device__ __forceinline__ T opaque(T v) {
    asm volatile("" : "+s"(v));
    return v;
}

// A value that is the same in every lane, made known to be so.
__device__ __forceinline__ double uniform_d(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readfirstlane((int)(x & 0xffffffffll));
    const int hi = __builtin_amdgcn_readfirstlane((int)(x >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Keeps the compiler from moving LDS loads across this point.  The loads of
// one step use fixed LDS addresses, so without it the loads of all steps of
// an unrolled loop would be issued together and take every register.
__device__ __forceinline__ void step_fence() { asm volatile("" ::: "memory"); }

// The same for a per-lane value: the lane and row predicates of the column
// steps (32 of them, one per step) are then formed in each panel instead of
// once for the whole kernel.
__device__ __forceinline__ int opaque_v(int v) {
    asm volatile("" : "+v"(v));
    return v;
}

__global__ __launch_bounds__(kThreads) void getrf_wide_kernel(WideParams P) {
    const int bm = P.b0 + int(blockIdx.y);
    double *__restrict__ AB = P.AB + int64_t(bm) * P.strideAB;
    int32_t *__restrict__ ipiv = P.ipiv + int64_t(bm) * P.strideP;
    int32_t *info = P.info + bm;
    char *scr = P.scratch + int64_t(blockIdx.y) * P.scratch_stride;
    int *counter = reinterpret_cast<int *>(scr);
    int *failed = counter + 1;
    int *solved = counter + 2;  // panels the forward substitution has applied
    char *slots = scr + kHdrBytes;
    const int n = P.n, kl = P.kl, ku = P.ku, kv = kl + ku, G = P.G;
    const int64_t ldab = P.ldab;
    const int t = threadIdx.x, wv = t >> 6;
    // window row of this thread in the factorisation (-1: none)
    const int myr0 = wv == 0 ? ((t & 63) < NB ? (t & 63) : -1) : NB + (wv - 1) * 64 + (t & 63);

    __shared__ double W[PR * LDW];
    __shared__ double sL11[NB * LDW];
    __shared__ double sU[NB * LDU];
    __shared__ double sA[NB * (PR - NB)];  // the applied panel's -L21, column-major
    __shared__ double sK[kWaves];
    __shared__ int sI[kWaves];
    __shared__ int s_perm[PR];
    __shared__ int s_p[NB];
    __shared__ int s_ok, s_ident, s_viol;

    // wait until panel k is published; false if the hand-off failed
    auto wait_panel = [&](int k) -> bool {
        if (t == 0) {
            int ok = 1;
            unsigned spins = 0;
            while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <= k) {
                if (__hip_atomic_load(failed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                    ok = 0;
                    break;
                }
                if (++spins > P.spin_limit) {
                    __hip_atomic_store(failed, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(info, INT_MIN, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    ok = 0;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            s_ok = ok;
        }
        __syncthreads();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        return s_ok != 0;
    };

    // ------------------------------------------ forward substitution --
    // L y = P b, the first half of the solve, trails the chain of panels in a
    // workgroup of its own: for each published panel it applies the panel's
    // net interchange, then y_top = L11^-1 b_top, then b_rest += (-L21) y_top
    // to a window of 288 rows of the right-hand sides (row r of column q at
    // W[prow(r) * LDW + q]).  Each value receives the fused multiply-adds of
    // the column steps in their order, with the multipliers of those steps,
    // so y is bitwise that of the unblocked forward pass.  It publishes how
    // many panels it has applied, and a panel's slot is rewritten only after
    // that (the owner of block b waits for panel b-G here before it factors).
    if (P.B != nullptr && int(blockIdx.x) == G) {
        double *Bm = P.B + int64_t(bm) * P.strideB;
        const int nr = P.nrhs;
        for (int idx = t; idx < PR * nr; idx += kThreads) {
            const int q = idx / PR, w = idx - q * PR;
            W[prow(w) * LDW + q] = w < n ? Bm[int64_t(q) * P.ldb + w] : 0.0;
        }
        __syncthreads();
        for (int k = 0; k < P.nblocks; ++k) {
            const int j0 = NB * k;
            const int Rw = min(NB + kl, n - j0);
            if (!wait_panel(k)) return;
            const char *slot = slots + size_t(k % G) * kSlotBytes;
            const int *sperm = reinterpret_cast<const int *>(slot);
            const double *gL11 = reinterpret_cast<const double *>(slot + kSlotInts * 4);
            const double *gNL = gL11 + NB * NB;
            if (!sperm[PR]) {
                // the panel's interchanges: one gather of whole rows
                for (int q0 = 0; q0 < nr; q0 += 8) {
                    double v[8];
                    const bool mv = t < Rw;
                    const int from = prow(j0 + (mv ? sperm[t] : 0)) * LDW;
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[q] = mv && q0 + q < nr ? W[from + q0 + q] : 0.0;
                    __syncthreads();
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (mv && q0 + q < nr) W[prow(j0 + t) * LDW + q0 + q] = v[q];
                    __syncthreads();
                }
            }
            // y_top = L11^-1 b_top, one thread per right-hand side (L11 unit
            // lower, column-major: L11(r, s) at [s * 32 + r])
            if (t < nr) {
                double y[NB];
#pragma unroll
                for (int r = 0; r < NB; ++r) y[r] = W[prow(j0 + r) * LDW + t];
#pragma unroll
                for (int s2 = 0; s2 < NB - 1; ++s2)
#pragma unroll
                    for (int r = s2 + 1; r < NB; ++r) y[r] = __builtin_fma(-gL11[s2 * NB + r], y[s2], y[r]);
#pragma unroll
                for (int r = 0; r < NB; ++r) W[prow(j0 + r) * LDW + t] = y[r];
            }
            __syncthreads();
            // rows 32..Rw-1 += (-L21) y_top, the steps in order
            for (int idx = t; idx < (PR - NB) * nr; idx += kThreads) {
                const int q = idx / (PR - NB), i = idx - q * (PR - NB);
                if (NB + i < Rw) {
                    double *bp = &W[prow(j0 + NB + i) * LDW + q];
                    double acc = *bp;
                    const int top = prow(j0) * LDW + q;
#pragma unroll 8
                    for (int s2 = 0; s2 < NB; ++s2)
                        acc = __builtin_fma(gNL[s2 * (PR - NB) + i], W[top + s2 * LDW], acc);
                    *bp = acc;
                }
            }
            __syncthreads();
            // rows j0..j0+31 are final; rows j0+288..j0+319 enter in their place
            for (int idx = t; idx < NB * nr; idx += kThreads) {
                const int q = idx / NB, i = idx - q * NB;
                const int r = j0 + i;
                double *wp = &W[prow(r) * LDW + q];
                if (r < n) Bm[int64_t(q) * P.ldb + r] = *wp;
                *wp = r + PR < n ? Bm[int64_t(q) * P.ldb + r + PR] : 0.0;
            }
            __syncthreads();
            if (t == 0) __hip_atomic_store(solved, k + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
    }

    for (int b = blockIdx.x; b < P.nblocks; b += G) {
        const int cb = NB * b;
        const int k0 = max(0, b - P.nblk);
        // ------------------------------------------------ load the window --
        {
            const int r0 = NB * k0;
#pragma unroll 1
            for (int idx = opaque_v(t); idx < PR * NB; idx += kThreads) {
                const int c = idx / PR, w = idx - c * PR;
                const int r = r0 + w, col = cb + c;
                const int d = r - col;
                const bool ok = r < n && col < n && d <= kl && d >= -kv;
                W[prow(r) * LDW + c] = ok ? AB[int64_t(col) * ldab + (kv + d)] : 0.0;
            }
        }
        __syncthreads();

        // ------------------------------------------- apply panels k0..b-1 --
        for (int k = k0; k < b; ++k) {
            const int j0 = NB * k;
            const int Rw = min(NB + kl, n - j0);  // rows of the panel's window in the matrix
            // the 32 band rows that enter the window after this panel are
            // original data: their loads go out before the wait
            double nxt[4];
            {
                const int tt = opaque_v(t);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int idx = tt + u * kThreads;
                    const int c = idx / NB, rn = j0 + PR + (idx - c * NB), col = cb + c;
                    const int dn = rn - col;
                    const bool okn = idx < NB * NB && rn < n && col < n && dn <= kl && dn >= -kv;
                    nxt[u] = okn ? AB[int64_t(col) * ldab + (kv + dn)] : 0.0;
                }
            }
            if (!wait_panel(k)) return;
            const int lane = opaque_v(t & 63);
            const char *slot = slots + size_t(k % G) * kSlotBytes;
            const int *sperm = reinterpret_cast<const int *>(slot);
            const double *gL11 = reinterpret_cast<const double *>(slot + kSlotInts * 4);
            const double *gNL = gL11 + NB * NB;
            // wave 0 brings L11 and the interchange flag to LDS (one round trip)
            if (wv == 0) {
                double lv[NB * NB / 64];
#pragma unroll
                for (int u = 0; u < NB * NB / 64; ++u) lv[u] = gL11[lane + 64 * u];
                const int idf = sperm[PR];
#pragma unroll
                for (int u = 0; u < NB * NB / 64; ++u) {
                    const int i = lane + 64 * u;
                    sL11[(i % NB) * LDW + (i / NB)] = lv[u];
                }
                if (lane == 0) s_ident = idf;
            }
            __syncthreads();
            if (!s_ident) {
                // the panel's interchanges as one gather of whole rows, eight
                // columns at a time
                const bool mv = t < Rw;
                const double *from = W + prow(j0 + (mv ? sperm[t] : 0)) * LDW;
                double *to = W + prow(j0 + (mv ? t : 0)) * LDW;
#pragma unroll 1
                for (int c0 = 0; c0 < NB; c0 += 8) {
                    double v[8];
                    if (mv) {
#pragma unroll
                        for (int c = 0; c < 8; ++c) v[c] = from[c0 + c];
                    }
                    __syncthreads();
                    if (mv) {
#pragma unroll
                        for (int c = 0; c < 8; ++c) to[c0 + c] = v[c];
                    }
                    __syncthreads();
                }
            }
            // U12 = L11^-1 * (rows 0..31) on wave 0, one lane per column, while
            // waves 1..4 bring the panel's -L21 to LDS (16-byte pieces) for the
            // update that follows
            if (wv != 0) {
                const double2 *src = reinterpret_cast<const double2 *>(gNL);
                double2 *dst = reinterpret_cast<double2 *>(sA);
                constexpr int kPieces = (PR - NB) * NB / 2;
                // (every thread's 16 pieces in flight at once: one memory latency)
                static_assert(kPieces % (kThreads - 64) == 0, "whole rounds");
                const int i0 = opaque_v(t - 64);
                double2 v[kPieces / (kThreads - 64)];
#pragma unroll
                for (int u = 0; u < kPieces / (kThreads - 64); ++u) v[u] = src[i0 + u * (kThreads - 64)];
#pragma unroll
                for (int u = 0; u < kPieces / (kThreads - 64); ++u) dst[i0 + u * (kThreads - 64)] = v[u];
            }
            if (wv == 0 && lane < NB) {
                // rows j0..j0+31 are 32 consecutive physical rows (288 and
                // every window start are multiples of 32)
                double *const col = W + opaque(prow(j0) * LDW) + lane;
                // (a base the compiler cannot fold: every load below is then
                // this register plus an immediate offset, instead of an address
                // register of its own hoisted out of the loops)
                const double *const Lm = sL11 + opaque_v(0);
                double y[NB];
#pragma unroll
                for (int r = 0; r < NB; ++r) y[r] = col[r * LDW];
#pragma unroll
                for (int s = 0; s < NB - 1; ++s) {
                    // one step's 31-s factor loads issued together, then used
                    step_fence();
                    double lv[NB];
#pragma unroll
                    for (int r = s + 1; r < NB; ++r) lv[r] = Lm[r * LDW + s];
                    step_fence();
#pragma unroll
                    for (int r = s + 1; r < NB; ++r) y[r] = __builtin_fma(-lv[r], y[s], y[r]);
                }
#pragma unroll
                for (int r = 0; r < NB; ++r) col[r * LDW] = y[r];
            }
            __syncthreads();
            // rows 32..Rw-1 += (-L21) * U12 on the matrix cores, wave g (1..4)
            // on rows 64g-32..64g+31.  Operand lanes of v_mfma_f64_16x16x4f64:
            // A[lane % 16][lane / 16], B[lane / 16][lane % 16]; accumulator
            // element q of a lane is D[4q + lane / 16][lane % 16].
            if (wv >= 1) {
                const int R0 = NB + 64 * (__builtin_amdgcn_readfirstlane(wv) - 1);
                if (R0 < Rw) {
                    const int ln = lane & 15, lk = lane >> 4;
                    // A(i, 4kb + lk) of row tile rt is sA[(4kb + lk) * 256 + R0 - 32 + 16rt + ln]
                    const double *const av = sA + lk * (PR - NB) + (R0 - NB) + ln;
                    // the wave's 64 rows are two groups of 32 consecutive
                    // physical rows; U12 is the group of rows j0..j0+31
                    double *const g0 = W + opaque(prow(j0 + R0) * LDW) + lk * LDW + ln;
                    double *const g1 = W + opaque(prow(j0 + R0 + NB) * LDW) + lk * LDW + ln;
                    const double *const bu = W + opaque(prow(j0) * LDW) + lk * LDW + ln;
                    auto arow = [&](int rt, int q, int ct) __attribute__((always_inline)) -> double * {
                        return (rt < 2 ? g0 : g1) + (16 * (rt & 1) + 4 * q) * LDW + 16 * ct;
                    };
                    v4d acc[4][2];
#pragma unroll
                    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                            for (int q = 0; q < 4; ++q) acc[rt][ct][q] = *arow(rt, q, ct);
#pragma unroll
                    for (int kb = 0; kb < NB / 4; ++kb) {
                        const double b0 = bu[4 * kb * LDW];
                        const double b1 = bu[4 * kb * LDW + 16];
#pragma unroll
                        for (int rt = 0; rt < 4; ++rt) {
                            const double a = av[4 * kb * (PR - NB) + 16 * rt];
                            acc[rt][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b0, acc[rt][0], 0, 0, 0);
                            acc[rt][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b1, acc[rt][1], 0, 0, 0);
                        }
                    }
#pragma unroll
                    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const int w = R0 + 16 * rt + 4 * q + lk;
                                if (w < Rw) *arow(rt, q, ct) = acc[rt][ct][q];
                            }
                }
            }
            __syncthreads();
            // rows j0..j0+31 are final: write them back; the rows that enter
            // the window (loaded above) take their physical rows
            {
                const int tt = opaque_v(t);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int idx = tt + u * kThreads;
                    if (idx < NB * NB) {
                        const int c = idx / NB, i = idx - c * NB;
                        const int col = cb + c;
                        const int r = j0 + i, d = r - col;
                        double *wp = &W[prow(r) * LDW + c];
                        if (r < n && col < n && d >= -kv) AB[int64_t(col) * ldab + (kv + d)] = *wp;
                        *wp = nxt[u];
                    }
                }
            }
            __syncthreads();
        }

        // ------------------------------------------------ factor panel b --
        // (with the fused forward substitution: the slot this panel takes is
        // free once that workgroup has applied panel b-G)
        if (P.B != nullptr && b >= G) {
            if (t == 0) {
                unsigned spins = 0;
                while (__hip_atomic_load(solved, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < b - G + 1) {
                    if (__hip_atomic_load(failed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
                    if (++spins > P.spin_limit) {
                        __hip_atomic_store(failed, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        __hip_atomic_store(info, INT_MIN, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            __syncthreads();
        }
        const int j0 = cb;
        const int nbn = min(NB, n - j0);
        const int Rn = min(nbn + kl, n - j0);
        const int myr = opaque_v(myr0);
        const int lane = opaque_v(t & 63);
        const bool own = myr >= 0 && myr < Rn;
        char *slot = slots + size_t(b % G) * kSlotBytes;
        int *gperm = reinterpret_cast<int *>(slot);
        double *gL11 = reinterpret_cast<double *>(slot + kSlotInts * 4);
        double *gNL = gL11 + NB * NB;
        const int mp = prow(j0 + max(myr, 0)) * LDW;
        double x[NB];
#pragma unroll
        for (int c = 0; c < NB; ++c) x[c] = own ? W[mp + c] : 0.0;

        // ---- first attempt: every pivot on the diagonal.  Partial pivoting
        // keeps the diagonal entry exactly when no candidate below it has a
        // larger pivot key (a tie goes to the first, the diagonal), so every
        // row checks itself at every step instead of taking part in an argmax.
        // Wave 0 (rows 0..31, row s in lane s) runs the 32 steps, lane s
        // publishing pivot row s in LDS; waves 1..4 apply each group of steps
        // while wave 0 computes the next.  The operations are those of the
        // pivoting loop below, so whenever it would not interchange, the
        // results are its results.
        bool viol = false;
        int finfo = 0;
        unsigned zmask = 0;  // columns whose pivot is zero
        if (t == 0) s_viol = 0;
        double r = 1.0 / x[0];  // wave 0: reciprocal of this row's entry in the next step's column
        double *const sUb = sU + opaque_v(0);  // (see the substitution above)
        // apply step S to a row held in xr (its window row wr, kept if !ok)
        auto upd_row = [&](double (&xr)[NB], int wr, bool ok, const double *us, int S, double piv,
                           double rcp, int km) __attribute__((always_inline)) {
            // the pivot row's entries issued together, then used
            double u[NB];
#pragma unroll
            for (int c = S + 1; c < NB; ++c) u[c] = us[c];
            step_fence();
            const int tt = wr - S;
            const bool cand = ok & (tt >= 1) & (tt <= km);
            viol |= cand && pivot_key(xr[S], tt) > pivot_key(piv, 0);
            // (a pivot below DBL_MIN divides instead of multiplying by its
            // reciprocal: that rare case is left to the pivoting path)
            viol |= piv != 0.0 && fabs(piv) < DBL_MIN;
            if (piv != 0.0 && cand) {
                const double l = xr[S] * rcp;
                xr[S] = l;
#pragma unroll
                for (int c = S + 1; c < NB; ++c) xr[c] = __builtin_fma(-l, u[c], xr[c]);
            }
        };
        // step S in wave 0: lane S's row is final; it writes the row and its
        // reciprocal to row S of sU (the buffer waves 1..4 read after the
        // group's barrier; one 8-byte store per entry, straight from its
        // register, as a paired store would first copy both into adjacent
        // registers), and every lane reads the row back at once (the LDS
        // operations of one wave complete in order).  The pivot and its
        // reciprocal come from lane S by lane reads instead (uniform, so the
        // branches on them are scalar; no LDS round trip on the chain).
        auto step_w0 = [&]<int S>() __attribute__((always_inline)) {
            if (S >= nbn) return;
            step_fence();
            double *us = sUb + S * LDU;
            if (lane == S) {
#pragma unroll
                for (int c = S; c < NB; ++c) {
                    us[c] = x[c];
                    step_fence();
                }
                us[NB] = r;
            }
            __builtin_amdgcn_wave_barrier();
            const double piv = readlane_d(x[S], S);
            const double rcp = readlane_d(r, S);
            const int km = min(kl, n - 1 - (j0 + S));
            upd_row(x, myr, own, us, S, piv, rcp, km);
            if (piv == 0.0) {
                zmask |= 1u << S;
                if (finfo == 0) finfo = j0 + S + 1;
            }
            if constexpr (S + 1 < NB) r = 1.0 / x[S + 1];
        };
        auto step_wk = [&]<int S>() __attribute__((always_inline)) {
            if (S >= nbn) return;
            step_fence();
            const double *us = sUb + S * LDU;
            const double piv = uniform_d(us[S]);
            const double rcp = uniform_d(us[NB]);
            const int km = min(kl, n - 1 - (j0 + S));
            upd_row(x, myr, own, us, S, piv, rcp, km);
            if (piv == 0.0) {
                zmask |= 1u << S;
                if (finfo == 0) finfo = j0 + S + 1;
            }
        };
        // groups of steps S0..S0+CNT-1; the last groups are short, so that
        // waves 1..4 (one group behind wave 0) finish soon after wave 0
        auto group_w0 = [&]<int S0, int CNT>() __attribute__((always_inline)) {
            if (S0 >= nbn) return;
            [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
                (step_w0.template operator()<S0 + Q>(), ...);
            }(std::make_integer_sequence<int, CNT>{});
            lds_barrier();
        };
        auto group_wk = [&]<int S0, int CNT>() __attribute__((always_inline)) {
            if (S0 >= nbn) return;
            lds_barrier();
            [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
                (step_wk.template operator()<S0 + Q>(), ...);
            }(std::make_integer_sequence<int, CNT>{});
        };
        static_assert(NB == 32, "groups of 8, 8, 8, 4, 2 and 2 steps");
        // no interchange: pivots, multipliers and U stay in place.  Each row
        // writes its part of the published L from its registers, and goes
        // back to its row of the window, from where all threads write the
        // panel's band entries with coalesced stores after the hand-over (one
        // LDS read and one store per entry: few registers).
        // (Done in both branches below, so that the rows' registers are not
        // carried across their join.)
        auto commit_spec = [&]() __attribute__((always_inline)) {
            if (myr >= 0) {
                // the published L straight from the registers, one store per
                // column (consecutive rows: consecutive addresses): L11 for
                // rows 0..31, -L21 below; zero-pivot columns, columns past
                // the matrix and rows outside it contribute zeros.  (Issued
                // first: the hand-over waits for them; the copy to the window
                // below goes on while they drain.)
                const unsigned zm = __builtin_amdgcn_readfirstlane(zmask);
#pragma unroll
                for (int sc = 0; sc < NB; ++sc) {
                    const bool live = myr < Rn && sc < nbn && !((zm >> sc) & 1u);
                    if (myr < NB)
                        gL11[sc * NB + myr] = (live && sc < myr) ? x[sc] : 0.0;
                    else
                        gNL[sc * (PR - NB) + (myr - NB)] = live ? -x[sc] : 0.0;
                }
#pragma unroll
                for (int c = 0; c < NB; ++c) W[mp + c] = x[c];
            }
            if (t < nbn) ipiv[j0 + t] = j0 + t + 1;
            if (t == 0) {
                gperm[PR] = 1;
                if (finfo != 0 && *info == 0) *info = finfo;
            }
        };
        // (after the barrier that follows commit_spec)
        // the band entries of the panel's columns, column by column: no other
        // workgroup reads them, so they are written after the hand-over (the
        // release fence of the hand-over then waits for, and writes back, only
        // the published L)
        auto commit_band = [&]() __attribute__((always_inline)) {
            const int tt = opaque_v(t);
#pragma unroll 1
            for (int idx = tt; idx < NB * PR; idx += kThreads) {
                const int c = idx / PR, w = idx - c * PR;
                const int d = w - c;
                if (c < nbn && w < Rn && d >= -kv && d <= kl)
                    AB[int64_t(j0 + c) * ldab + (kv + d)] = W[prow(j0 + w) * LDW + c];
            }
        };
        bool spec_ok;
        if (__builtin_amdgcn_readfirstlane(wv) == 0) {
            group_w0.template operator()<0, 8>();
            group_w0.template operator()<8, 8>();
            group_w0.template operator()<16, 8>();
            group_w0.template operator()<24, 4>();
            group_w0.template operator()<28, 2>();
            group_w0.template operator()<30, 2>();
            if (__ballot(viol) && lane == 0) s_viol = 1;
            lds_barrier();
            spec_ok = s_viol == 0;
            if (spec_ok) commit_spec();
        } else {
            group_wk.template operator()<0, 8>();
            group_wk.template operator()<8, 8>();
            group_wk.template operator()<16, 8>();
            group_wk.template operator()<24, 4>();
            group_wk.template operator()<28, 2>();
            group_wk.template operator()<30, 2>();
            if (__ballot(viol) && lane == 0) s_viol = 1;
            lds_barrier();
            spec_ok = s_viol == 0;
            if (spec_ok) commit_spec();
        }
        if (!spec_ok) {
            // ---- partial pivoting, in the window in LDS: one thread per row,
            // whole rows interchanged (so the window ends with L in its final
            // row order, as the blocks it updates need it), four barriers per
            // column step.  This path runs only for panels that interchange
            // rows, and keeps few values in registers.
            const int wvu = __builtin_amdgcn_readfirstlane(wv);
            const int myr = opaque_v(myr0);
            const bool own = myr >= 0 && myr < Rn;
            double *const row1 = W + prow(j0 + max(myr, 0)) * LDW;
            for (int i = t; i < PR; i += kThreads) s_perm[i] = i;
            int pinfo = 0;
            unsigned pz = 0;
            __syncthreads();
#pragma unroll 1
            for (int jj = 0; jj < nbn; ++jj) {
                const int col = j0 + jj;
                const int km = min(kl, n - 1 - col);
                const int tt = myr - jj;
                const bool cand = own & (tt >= 0) & (tt <= km);
                const double key = cand ? pivot_key(row1[jj], tt) : -2.0;
                const double wmax = wave_max_d(key);
                // rows are in lane order inside a wave: the lowest lane with
                // the largest key is the first such row
                const unsigned long long hit = __ballot(key == wmax);
                const int f = __builtin_amdgcn_readfirstlane(__builtin_ctzll(hit));
                const int frow = __builtin_amdgcn_readlane(myr, f);
                if (lane == 0) {
                    sK[wvu] = wmax;
                    sI[wvu] = wmax > -2.0 ? frow : INT_MAX;
                }
                __syncthreads();
                double bk = sK[0];
                int bi = sI[0];
#pragma unroll
                for (int w2 = 1; w2 < kWaves; ++w2) {
                    const double kw = sK[w2];
                    const int iw = sI[w2];
                    const bool bt = key_better(kw, iw, bk, bi);
                    bk = bt ? kw : bk;
                    bi = bt ? iw : bi;
                }
                const int p = bi - jj;  // uniform
                double *const prow_j = W + prow(col) * LDW;
                double *const prow_p = W + prow(col + p) * LDW;
                const double piv = prow_p[jj];
                if (t == 0) {
                    ipiv[col] = col + p + 1;
                    s_p[jj] = p;
                }
                const bool elim = piv != 0.0;
                if (!elim) {
                    pz |= 1u << jj;
                    if (pinfo == 0) pinfo = col + 1;
                }
                __syncthreads();
                if (elim && p != 0) {
                    if (t < NB) {
                        const double a0 = prow_j[t];
                        prow_j[t] = prow_p[t];
                        prow_p[t] = a0;
                    } else if (t == NB) {
                        const int a0 = s_perm[jj];
                        s_perm[jj] = s_perm[jj + p];
                        s_perm[jj + p] = a0;
                    }
                }
                __syncthreads();
                if (elim && own && tt >= 1 && tt <= km) {
                    const double l = fabs(piv) >= DBL_MIN ? row1[jj] * (1.0 / piv) : row1[jj] / piv;
                    row1[jj] = l;
#pragma unroll 1
                    for (int c = jj + 1; c < NB; ++c) row1[c] = __builtin_fma(-l, prow_j[c], row1[c]);
                }
                __syncthreads();
            }
            // the band: U rows and the multipliers in product form (each in
            // the row its data row had when its column was eliminated, found
            // by replaying the interchanges from the data row's first place)
            if (own) {
                int pos = s_perm[myr];
#pragma unroll 1
                for (int jj = 0; jj < nbn; ++jj) {
                    const int col = j0 + jj;
                    const int p = s_p[jj];
                    if (!((pz >> jj) & 1u) && p != 0)
                        pos = pos == jj ? jj + p : (pos == jj + p ? jj : pos);
                    const int km = min(kl, n - 1 - col);
                    if (pos > jj && pos - jj <= km)
                        AB[int64_t(col) * ldab + (kv + pos - jj)] = row1[jj];
                }
#pragma unroll 1
                for (int c = myr; c < nbn; ++c)
                    if (myr - c >= -kv) AB[int64_t(j0 + c) * ldab + (kv + myr - c)] = row1[c];
            }
            // the panel's L in its final row order for the blocks it updates
            if (myr >= 0) {
                gperm[myr] = s_perm[myr];
                if (myr < NB) {
#pragma unroll 1
                    for (int s2 = 0; s2 < NB; ++s2)
                        gL11[s2 * NB + myr] = (own && s2 < myr && !((pz >> s2) & 1u)) ? row1[s2] : 0.0;
                } else {
#pragma unroll 1
                    for (int s2 = 0; s2 < NB; ++s2)
                        gNL[s2 * (PR - NB) + myr - NB] =
                            (own && s2 < nbn && !((pz >> s2) & 1u)) ? -row1[s2] : 0.0;
                }
            }
            if (t == 0) {
                gperm[PR] = 0;
                if (pinfo != 0 && *info == 0) *info = pinfo;
            }
        }
        static_assert(NB + (kWaves - 1) * 64 == PR, "one thread per window row");
        // publish the panel
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __syncthreads();
        if (t == 0) __hip_atomic_store(counter, b + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (spec_ok) {
            commit_band();
            __syncthreads();  // the window is loaded again next
        }
    }
}

// in-matrix fill slots (band rows 0..kl-1) start at zero, info at 0, and the
// hand-off counters of the launch's matrices at 0
__global__ void wide_init_kernel(double *ABbase, int64_t ldab, int64_t strideAB, int32_t *info,
                                 char *scratch, int64_t scratch_stride, int n, int kl, int ku,
                                 int b0, int count) {
    const int kv = kl + ku;
    const int64_t total = int64_t(n) * kl;
    for (int m = blockIdx.y; m < count; m += gridDim.y) {
        double *AB = ABbase + int64_t(b0 + m) * strideAB;
        for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
             e += int64_t(gridDim.x) * blockDim.x) {
            const int64_t c = e / kl, r = e - c * kl;
            if (r >= kv - c) AB[c * ldab + r] = 0.0;
        }
        if (blockIdx.x == 0 && threadIdx.x < 3) {
            if (threadIdx.x == 0) info[b0 + m] = 0;
            reinterpret_cast<int *>(scratch + int64_t(m) * scratch_stride)[threadIdx.x] = 0;
        }
    }
}

struct WideGeom {
    int nblk, G, nblocks;
};

WideGeom wide_geom(int64_t n, int64_t kl, int64_t ku) {
    WideGeom g;
    g.nblk = int((kl + ku + NB - 1) / NB);
    g.nblocks = int((n + NB - 1) / NB);
    g.G = std::max(1, std::min(g.nblk + 1, g.nblocks));
    return g;
}

// workgroups of the kernel that can be resident at once on the current device
int max_resident_groups() {
    static int cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
    if (cached[dev] <= 0) {
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, getrf_wide_kernel, kThreads, 0) !=
                hipSuccess ||
            per_cu < 1)
            per_cu = 1;
        cached[dev] = per_cu * device_cu_count();
    }
    return cached[dev];
}

unsigned spin_limit() {
    // polls of a bounded wait before the hand-off is declared failed (each
    // poll is a device-scope load and a short sleep: about 4 s in all)
    static unsigned cached = 0;
    if (cached == 0) {
        cached = 1u << 22;
        if (const char *e = std::getenv("BANDLU_WIDE_SPIN_LIMIT")) cached = (unsigned)std::strtoul(e, nullptr, 10);
        if (cached == 0) cached = 1;
    }
    return cached;
}

}  // namespace

bool getrf_wide_fits(int64_t n, int64_t kl, int64_t ku, int64_t batch) {
    if (kl > kMaxKl || n > kMaxN || batch < 1) return false;
    const WideGeom g = wide_geom(n, kl, ku);
    return g.G <= max_resident_groups();
}

// whether the whole batch fits one launch of co-resident workgroups
bool getrf_wide_one_launch(int64_t n, int64_t kl, int64_t ku, int64_t batch) {
    if (!getrf_wide_fits(n, kl, ku, batch)) return false;
    return int64_t(wide_geom(n, kl, ku).G) * batch <= max_resident_groups();
}

// one matrix with the forward substitution fused: G + 1 co-resident
// workgroups, and at most LDW right-hand sides in the window
bool getrf_wide_fused_fits(int64_t n, int64_t kl, int64_t ku, int64_t nrhs) {
    if (kl > kMaxKl || n > kMaxN || nrhs < 1 || nrhs > LDW) return false;
    return wide_geom(n, kl, ku).G + 1 <= max_resident_groups();
}

// matrices per launch (the matrices of a launch share the scratch)
static int64_t wide_chunk(int64_t n, int64_t kl, int64_t ku, int64_t batch, int extra = 0) {
    const WideGeom g = wide_geom(n, kl, ku);
    return std::max<int64_t>(1, std::min<int64_t>(batch, max_resident_groups() / (g.G + extra)));
}

static int64_t wide_matrix_bytes(int64_t n, int64_t kl, int64_t ku) {
    const WideGeom g = wide_geom(n, kl, ku);
    return kHdrBytes + int64_t(g.G) * int64_t(kSlotBytes);
}

size_t getrf_wide_scratch_bytes(int64_t n, int64_t kl, int64_t ku, int64_t batch) {
    return size_t(wide_chunk(n, kl, ku, batch) * wide_matrix_bytes(n, kl, ku));
}

int launch_getrf_wide(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s, void *scratch, size_t scratch_bytes,
                      double *dB, int64_t ldb, int64_t strideB, int64_t nrhs) {
    const int extra = dB != nullptr ? 1 : 0;
    if (!getrf_wide_fits(n, kl, ku, batch) ||
        (extra && !getrf_wide_fused_fits(n, kl, ku, nrhs))) {
        set_error("band_getrf: the persistent wide-band variant needs kl <= %d and "
                  "(kl+ku+31)/32 + 1 co-resident workgroups (one more, and at most %d "
                  "right-hand sides, with the fused forward substitution)", kMaxKl, LDW);
        return BANDLU_ERR_UNSUPPORTED;
    }
    const WideGeom g = wide_geom(n, kl, ku);
    int64_t chunk = wide_chunk(n, kl, ku, batch, extra);
    const int64_t per = wide_matrix_bytes(n, kl, ku);
    bool own_alloc = false;
    if (scratch == nullptr) {
        if (hipError_t e = hipMallocAsync(&scratch, size_t(chunk * per), s); e != hipSuccess)
            return hip_fail(e, "band_getrf (wide-band scratch)");
        own_alloc = true;
    } else {
        // a caller's buffer: as many matrices per launch as it holds (the
        // launches of a batch run one after another on the stream and reuse it)
        if (scratch_bytes < size_t(per)) {
            set_error("band_getrf: the wide-band variant needs %lld bytes of scratch per matrix "
                      "for kl = %lld, ku = %lld; %zu available",
                      (long long)per, (long long)kl, (long long)ku, scratch_bytes);
            return BANDLU_ERR_UNSUPPORTED;
        }
        chunk = std::min<int64_t>(chunk, int64_t(scratch_bytes / size_t(per)));
    }
    WideParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.info = d_info;
    P.scratch = static_cast<char *>(scratch);
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    P.scratch_stride = per;
    P.n = (int)n;
    P.kl = (int)kl;
    P.ku = (int)ku;
    P.nblk = g.nblk;
    P.G = g.G;
    P.nblocks = g.nblocks;
    P.spin_limit = spin_limit();
    P.B = dB;
    P.ldb = ldb;
    P.strideB = strideB;
    P.nrhs = (int)nrhs;
    int rc = BANDLU_OK;
    for (int64_t b0 = 0; b0 < batch; b0 += chunk) {
        const int cnt = (int)std::min<int64_t>(chunk, batch - b0);
        const int64_t total = n * kl;
        const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 1024));
        hipLaunchKernelGGL(wide_init_kernel, dim3(gx, (unsigned)std::min(cnt, 65535)), dim3(256), 0, s,
                           dAB, ldab, strideAB, d_info, P.scratch, per, (int)n, (int)kl, (int)ku,
                           (int)b0, cnt);
        if (hipError_t e = hipGetLastError(); e != hipSuccess) {
            rc = hip_fail(e, "band_getrf (wide-band init)");
            break;
        }
        P.b0 = (int)b0;
        void *args[] = {&P};
        if (hipError_t e = hipLaunchCooperativeKernel((const void *)getrf_wide_kernel,
                                                      dim3((unsigned)(g.G + extra), (unsigned)cnt),
                                                      dim3(kThreads), args, 0, s);
            e != hipSuccess) {
            rc = hip_fail(e, "band_getrf (wide-band persistent kernel)");
            break;
        }
    }
    if (own_alloc) {
        if (hipError_t e = hipFreeAsync(scratch, s); e != hipSuccess && rc == BANDLU_OK)
            rc = hip_fail(e, "band_getrf (wide-band scratch release)");
    }
    return rc;
}

}  // namespace bandlu
