// Blocked banded LU with partial pivoting for wide bands (Sec. III-A's
// specialised algorithm f(N) when kl+ku is large): xGBTRF in panels of NB = 32
// columns, one launch per panel.
//
// Launch k covers the band columns that panel k-1 can still change (up to
// j0 + NB - 1 + kl + ku) in blocks of 32 columns, one workgroup per block and
// one thread per band row, the row's 32 entries held in registers:
//   phase A: the block receives panel k-1's row interchanges and rank-1
//            updates one step after another, in the unblocked order and over
//            the same columns (up to the update extent ju of each step, none
//            for a zero pivot), so every entry sees the same fused
//            multiply-adds as in the unblocked algorithm;
//   phase B: workgroup 0's block is panel k itself (its rows below panel
//            k-1's reach were loaded too); it is factored in place with
//            partial pivoting while the other workgroups finish their blocks.
// Rows are exchanged and the pivot row is broadcast through double-buffered
// LDS rows with one barrier per step.  Stream order between launches carries
// the panel-to-panel dependency.
#include <algorithm>
#include <cfloat>
#include <climits>

#include "bufio.hpp"
#include "common.hpp"
#include "wave.hpp"

namespace bandlu {

int launch_getrf_blocked(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                         int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                         int64_t batch, hipStream_t s);
int launch_band_zero_fill(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int64_t strideAB, int32_t *d_info, int64_t batch, hipStream_t s);

namespace {

constexpr int NB = 32;        // panel width
constexpr int NBC = 32;       // trailing block width
constexpr int kMaxKl = 256;   // one thread per row: NB + NB + kl <= 320 threads


// ------------------------------------------------------------- fused step --
// One launch per panel.  Workgroup x of the launch owns the 32 columns
// cb = jn + 32x .. of the band, one thread per row, the 32 entries of its row in
// registers.
//   phase A (has_update): apply the interchanges and rank-1 updates of panel
//     j0 = jn - NB to the block, step by step in the unblocked order;
//   phase B (workgroup 0, has_factor): the block is panel jn itself; factor it
//     with partial pivoting (its rows below the old panel were loaded too).
// Rows are exchanged and the pivot row broadcast through double-buffered LDS
// rows, one barrier per step.
constexpr int kRows = 320;  // threads: NB + NB + kl rows at most (kl <= 256)

struct StepParams {
    double *AB;
    int32_t *ipiv;
    int32_t *info;
    int64_t ldab, strideAB, strideP;
    int n, kl, ku;
    int j0;          // panel whose update is applied (has_update)
    int jn;          // first column of the blocks (= next panel when has_factor)
    int has_update, has_factor;
};

__global__ __launch_bounds__(kRows) void blk_step_kernel(StepParams P) {
    const int bmat = blockIdx.y;
    double *__restrict__ AB = P.AB + int64_t(bmat) * P.strideAB;
    int32_t *__restrict__ ipiv = P.ipiv + int64_t(bmat) * P.strideP;
    const int n = P.n, kl = P.kl, ku = P.ku, kv = kl + ku;
    const int64_t ldab = P.ldab;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const bool upd = P.has_update != 0;
    const bool fac = P.has_factor != 0 && blockIdx.x == 0;
    const int j0 = P.j0, jn = P.jn;
    const int nb = upd ? min(NB, n - j0) : 0;          // width of the applied panel
    const int nbn = min(NB, n - jn);                   // width of the next panel
    const int rb = upd ? j0 : jn;                      // first row held
    const int cb = jn + blockIdx.x * NBC;              // first column held
    int clast = upd ? min(n - 1, j0 + nb - 1 + kv) : jn + nbn - 1;
    if (fac) clast = max(clast, jn + nbn - 1);  // the factored block spans the whole next panel
    const int W = min(NBC, clast - cb + 1);
    int rows = (upd ? nb + kl : 0);
    if (fac) rows = (upd ? nb : 0) + nbn + kl;
    rows = min(rows, n - rb);
    const int r = rb + t;                              // matrix row of this thread
    const bool own = t < rows;

    __shared__ double S[2][NBC];
    __shared__ double T2[2][NBC];
    __shared__ double s_key[kRows / 64];
    __shared__ int s_idx[kRows / 64];
    __shared__ double s_val[kRows / 64];
    __shared__ int s_piv[NB];
    __shared__ int s_nz[NB];   // applied panel: pivot of the step is nonzero
    __shared__ int s_ju[NB];   // applied panel: update extent of the step
    __shared__ int s_jub;      // factored panel: update extent before it

    double x[NBC];
    unsigned okx = 0;
#pragma unroll
    for (int c = 0; c < NBC; ++c) {
        const int col = cb + c;
        const bool ok = own & (c < W) & (col - r <= kv) & (r - col <= kl);
        okx |= unsigned(ok) << c;
        x[c] = ld_clamped(AB, int64_t(col) * ldab + (kv + r - col), ok);
    }
#pragma unroll
    for (int c = 0; c < NBC; ++c) x[c] = keep_if(x[c], okx, c);
    int step = 0;  // parity of the LDS row buffers

    // ---------------------------------------------------------- phase A --
    // Update extent (xGBTRF's ju): step j updates columns j+1..ju_j with
    // ju_j = max(ju_{j-1}, min(j+ku+p_j, n-1)) over the steps with a nonzero
    // pivot.  At such a step ju_j equals the maximum of min(s+ku+p_s, n-1) over
    // s = j-kl..j whatever the pivots of those s were: a step s < j-kl reaches
    // at most s+kl+ku < j+ku, and a zero-pivot step s < j has p_s = 0 and
    // reaches s+ku < j+ku.  So the extent follows from the last kl+1 pivots.
    auto reach = [&](int s) -> int {
        return s < 0 ? 0 : min(s + ku + (ipiv[s] - 1 - s), n - 1);
    };
    if (upd) {
        // the panel's pivots, staged once, with each step's extent and whether
        // its pivot (the final diagonal entry) is nonzero
        __shared__ int s_c[kRows];
        if (t < kl + nb) s_c[t] = reach(j0 - kl + t);
        if (t < nb) {
            s_piv[t] = ipiv[j0 + t] - 1 - (j0 + t);
            s_nz[t] = AB[int64_t(j0 + t) * ldab + kv] != 0.0;
        }
        lds_barrier();
        if (t < nb) {
            int m = 0;
            for (int u = 0; u <= kl + t; ++u) m = max(m, s_c[u]);
            s_ju[t] = m;
        }
        // multiplier of panel column jj for this thread's row, loaded 4 steps
        // ahead (only used by rows that have one: no need to clear the others)
        auto lval = [&](int jj) -> double {
            const int j = j0 + jj;
            const int tt = t - jj;
            const bool ok = own & (jj < nb) & (tt >= 1) & (tt <= min(kl, n - 1 - j));
            return ld_clamped(AB, int64_t(j) * ldab + (kv + tt), ok);
        };
        double lr[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) lr[q] = lval(q);
        lds_barrier();
#pragma unroll 1
        for (int j4 = 0; j4 < nb; j4 += 4) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int jj = j4 + q;
                if (jj < nb) {
                    const int j = j0 + jj;
                    const int p = s_piv[jj];
                    const int km = min(kl, n - 1 - j);
                    const bool nz = s_nz[jj] != 0;
                    const int ncol = s_ju[jj] - cb;  // block columns c < ncol are within ju
                    const double l = lr[q];
                    lr[q] = lval(jj + 4);
                    const int A = step & 1;
                    ++step;
                    if (t == jj + p) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) S[A][c] = x[c];
                    }
                    if (p != 0 && t == jj) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) T2[A][c] = x[c];
                    }
                    lds_barrier();
                    // (a zero pivot has p = 0: no interchange and no update)
                    if (t == jj) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) if (c <= ncol) x[c] = S[A][c];
                    } else if (p != 0 && t == jj + p) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) if (c <= ncol) x[c] = T2[A][c];
                    }
                    if (nz && t > jj && t - jj <= km) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c)
                            if (c <= ncol) x[c] = __builtin_fma(-l, S[A][c], x[c]);
                    }
                }
            }
        }
    }
    // ---------------------------------------------------------- phase B --
    if (fac) {
        const int off = upd ? nb : 0;  // thread index of row jn
        int info = 0;
        // extent before the panel, from the kl steps before it
        if (t == 0) s_jub = 0;
        lds_barrier();
        if (t < kl && jn - 1 - t >= 0) atomicMax(&s_jub, reach(jn - 1 - t));
        lds_barrier();
        int ju = s_jub;
#pragma unroll
        for (int jj = 0; jj < NB; ++jj) {
            if (jj < nbn) {
                const int j = jn + jj;
                const int km = min(kl, n - 1 - j);
                const int tt = t - off - jj;  // candidate index of this row
                const double v = x[jj];
                double key = (own && tt >= 0 && tt <= km)
                                 ? (__builtin_isnan(v) ? (tt == 0 ? __builtin_inf() : -1.0) : fabs(v))
                                 : -2.0;
                // wave max by DPP inside rows of 16 lanes, then across the 4 rows;
                // rows are in lane order, so the lowest matching lane is the first index
                double km16 = key;
                km16 = fmax(km16, dpp_d<0xB1>(km16));   // quad_perm [1,0,3,2]
                km16 = fmax(km16, dpp_d<0x4E>(km16));   // quad_perm [2,3,0,1]
                km16 = fmax(km16, dpp_d<0x141>(km16));  // row_half_mirror
                km16 = fmax(km16, dpp_d<0x140>(km16));  // row_mirror
                const double wmax = fmax(fmax(readlane_d(km16, 0), readlane_d(km16, 16)),
                                         fmax(readlane_d(km16, 32), readlane_d(km16, 48)));
                const unsigned long long hit = __ballot(key == wmax);
                const int first = __builtin_amdgcn_readfirstlane(__builtin_ctzll(hit));
                if (lane == 0) {
                    s_key[wv] = wmax;
                    s_idx[wv] = wv * 64 + first - off - jj;
                    s_val[wv] = readlane_d(v, first);
                }
                lds_barrier();
                double bk = s_key[0], bv = s_val[0];
                int bi = s_idx[0];
#pragma unroll
                for (int w = 1; w < kRows / 64; ++w)
                    if (key_better(s_key[w], s_idx[w], bk, bi)) { bk = s_key[w]; bi = s_idx[w]; bv = s_val[w]; }
                const int p = bi;
                if (t == 0) ipiv[j] = j + p + 1;
                const int A = step & 1;
                ++step;
                if (bv != 0.0) {
                    ju = max(ju, min(j + ku + p, n - 1));
                    const int ncol = ju - cb;
                    if (t == off + jj + p) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) S[A][c] = x[c];
                    }
                    if (p != 0 && t == off + jj) {
#pragma unroll
                        for (int c = 0; c < NBC; ++c) T2[A][c] = x[c];
                    }
                    lds_barrier();
                    // the interchange covers panel columns jj..; earlier columns
                    // keep their multipliers (product form of L)
                    if (t == off + jj) {
#pragma unroll
                        for (int c = jj; c < NBC; ++c) x[c] = c <= ncol ? S[A][c] : x[c];
                    } else if (p != 0 && t == off + jj + p) {
#pragma unroll
                        for (int c = jj; c < NBC; ++c) x[c] = c <= ncol ? T2[A][c] : x[c];
                    }
                    const double piv = S[A][jj];
                    if (tt >= 1 && tt <= km && own) {
                        const double l = fabs(piv) >= DBL_MIN ? x[jj] * (1.0 / piv) : x[jj] / piv;
                        x[jj] = l;
#pragma unroll
                        for (int c = jj + 1; c < NBC; ++c)
                            x[c] = c <= ncol ? __builtin_fma(-l, S[A][c], x[c]) : x[c];
                    }
                } else {
                    if (info == 0) info = j + 1;
                    lds_barrier();  // keep one barrier per step on every path
                }
            }
        }
        if (t == 0 && info != 0 && P.info[bmat] == 0) P.info[bmat] = info;
    }
    // -------------------------------------------------------- write back --
#pragma unroll
    for (int c = 0; c < NBC; ++c) {
        const int col = cb + c;
        if (own && c < W && col - r <= kv && r - col <= kl) AB[int64_t(col) * ldab + (kv + r - col)] = x[c];
    }
}

__global__ void zero_fill_kernel(double *ABbase, int64_t ldab, int64_t strideAB, int32_t *info,
                                 int n, int kl, int ku, int64_t batch) {
    // in-matrix fill slots (band rows 0..kl-1) start at zero; info starts at 0
    const int kv = kl + ku;
    const int64_t total = int64_t(n) * kl;
    for (int64_t b = blockIdx.y; b < batch; b += gridDim.y) {
        double *AB = ABbase + b * strideAB;
        for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
             e += int64_t(gridDim.x) * blockDim.x) {
            const int64_t c = e / kl, r = e - c * kl;
            if (r >= kv - c) AB[c * ldab + r] = 0.0;
        }
        if (blockIdx.x == 0 && threadIdx.x == 0) info[b] = 0;
    }
}

}  // namespace

int launch_band_zero_fill(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int64_t strideAB, int32_t *d_info, int64_t batch, hipStream_t s) {
    const int64_t total = n * kl;
    const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 4096));
    hipLaunchKernelGGL(zero_fill_kernel, dim3(gx, (unsigned)std::min<int64_t>(batch, 65535)),
                       dim3(256), 0, s, dAB, ldab, strideAB, d_info, (int)n, (int)kl, (int)ku, batch);
    BANDLU_CHECK_LAUNCH("band_getrf (fill-row init)");
    return BANDLU_OK;
}

int launch_getrf_blocked(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                         int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                         int64_t batch, hipStream_t s) {
    if (kl > kMaxKl || batch > 65535) {
        set_error("band_getrf: blocked variant needs kl <= %d", kMaxKl);
        return BANDLU_ERR_UNSUPPORTED;
    }
    if (int rc = launch_band_zero_fill(n, kl, ku, dAB, ldab, strideAB, d_info, batch, s)) return rc;
    const int kv = int(kl + ku);
    StepParams Q;
    Q.AB = dAB;
    Q.ipiv = d_ipiv;
    Q.info = d_info;
    Q.ldab = ldab;
    Q.strideAB = strideAB;
    Q.strideP = strideP;
    Q.n = (int)n;
    Q.kl = (int)kl;
    Q.ku = (int)ku;
    // launch 0 factors panel 0; launch k applies panel k-1 and factors panel k
    for (int64_t jn = 0; jn < n + NB; jn += NB) {
        Q.has_update = jn > 0;
        Q.j0 = (int)(jn - NB);
        Q.jn = (int)jn;
        Q.has_factor = jn < n;
        int64_t blocks = 1;
        if (Q.has_update) {
            const int64_t nb = std::min<int64_t>(NB, n - Q.j0);
            const int64_t clast = std::min<int64_t>(n - 1, Q.j0 + nb - 1 + kv);
            blocks = clast >= jn ? (clast - jn + 1 + NBC - 1) / NBC : 0;
        }
        if (blocks == 0) break;
        hipLaunchKernelGGL(blk_step_kernel, dim3((unsigned)blocks, (unsigned)batch), dim3(kRows),
                           0, s, Q);
        BANDLU_CHECK_LAUNCH("band_getrf (blocked step)");
    }
    return BANDLU_OK;
}

}  // namespace bandlu
