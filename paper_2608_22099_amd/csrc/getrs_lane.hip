// Band solve for narrow bands (kl + ku <= 63, ldab <= 64) with the band
// factors (xGBTRS, no transpose; the "lu(A) \ B" of Listings 1 and 2): one
// wavefront per right-hand side, every row of the active window in a lane of
// its own, so that a step is one fused multiply-add per lane and the chain
// from one row to the next is a lane read, that fused multiply-add and (in
// the backward pass) the division by the diagonal entry.
//
// Forward pass (L and the interchanges, rows j+1..j+kl): row r lives in lane
// r mod 64.  Step j applies the interchange of ipiv[j] (the two lanes
// exchange their values; the steps of a block of 64 that interchange are
// marked in a scalar mask), takes b(j) from its lane and updates
//   b(r) = fma(-l(r,j), b(j), b(r)),   r = j+1..j+min(kl, n-1-j).
// The lane of row j keeps b(j), now final, for one coalesced store per block
// and takes row j+64, loaded two blocks ahead.
// Backward pass (U with its kl+ku superdiagonals): the same with j descending,
//   x(j) = b(j) / u(j,j),  b(i) = fma(-u(i,j), x(j), b(i)),  i = j-kv..j-1,
// where every lane forms x(j) from the scalar b(j) and a broadcast LDS read of
// u(j,j).  The operations and their order per entry are those of the plain
// column-oriented loops, so the solution is bitwise theirs.
//
// The factor columns reach LDS in chunks of 32 columns (a ring of 64 columns,
// column c in slot c mod 64), one batch of 16-byte loads a chunk ahead; each
// lane reads its entry of a column two steps before the step needs it.  Steps
// issue no global memory operation.
#include "bufio.hpp"
#include "common.hpp"

#include <utility>

namespace bandlu {

int launch_getrs_lane(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s);
bool getrs_lane_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab);

namespace {

constexpr int kChunk = 32;  // factor columns per staged chunk

struct LaneParams {
    const double *AB;
    const int32_t *ipiv;
    double *B;
    int64_t ldab, strideAB, strideP, ldb, strideB;
    int n, kl, kv, nrhs;
};

__device__ __forceinline__ unsigned long long lane_low(int k) {
    return k >= 64 ? ~0ull : (1ull << k) - 1;
}

__device__ __forceinline__ unsigned long long lane_rotl(unsigned long long m, int k) {
    return k == 0 ? m : (m << k) | (m >> (64 - k));
}

// a lane index hidden from loop-invariant motion, so that what a step forms
// from it is formed in that step instead of 64 values being kept live across
// the loop
__device__ __forceinline__ int lane_opaque_v(int v) {
    asm volatile("" : "+v"(v));
    return v;
}

// lane mask constants, formed where they are used from an opaque 1 (as
// literals the optimiser keeps all of them live across the loop)
__device__ __forceinline__ unsigned long long lane_one() {
    unsigned long long o = 1;
    asm volatile("" : "+s"(o));
    return o;
}
__device__ __forceinline__ unsigned long long lane_bit(int q) { return lane_one() << q; }
__device__ __forceinline__ unsigned long long lane_below(int q) {  // lanes 0..q-1, 0 <= q <= 63
    const unsigned long long o = lane_one();
    return (o << q) - o;
}

// the mask of a step, formed where it is used (an opaque copy keeps the
// optimiser from hoisting all 64 rotations out of the loop)
__device__ __forceinline__ unsigned long long lane_mask(unsigned long long m, int k) {
    asm volatile("" : "+s"(m));
    return lane_rotl(m, k);
}

// BULK (kl + ku <= 32): a lane changes rows in two batches per block of 64
// steps (lanes 0-31, then 32-63), each with one coalesced store of the rows
// it finishes; wider bands change the lane of each pivot row at its step.
template <bool BULK>
__global__ __launch_bounds__(64) void getrs_lane_kernel(LaneParams P) {
    const int L = threadIdx.x;
    const int64_t sys = blockIdx.x / P.nrhs;
    const int64_t rhs = blockIdx.x - sys * P.nrhs;
    const int n = P.n, kl = P.kl, kv = P.kv, ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + sys * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    const Buf bb = make_buf(P.B + sys * P.strideB + rhs * P.ldb, uint32_t(n) * 8u);
    const Buf pb = make_buf(P.ipiv + sys * P.strideP, uint32_t(n) * 4u);
    // ring of 64 factor columns: column c in slot c mod 64, its entry of row r
    // at position r mod 64 (ldab <= 64 keeps them apart), so that the lane of
    // row r reads slot q at q*64 + L: an address with no per-step arithmetic
    __shared__ double ring[64 * 64];

    // chunk k = factor columns 32k..32k+31: lane t loads band row t of each
    double stg[kChunk];
    // (lanes past ldab and columns outside the matrix read out of range: the
    // offset, below 2^32 for every column a chunk names, gets the top bit by
    // arithmetic; a test there becomes a divergent branch around every load)
    const uint32_t lane_out = L < ldab ? 0u : kOutside;
    auto stage = [&](int k) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kChunk; ++q) {
            const int c = k * kChunk + q;
            const uint32_t out = lane_out | (((k >= 0) & (c < n)) ? 0u : kOutside);
            stg[q] = buf_ld(ab, (uint32_t(c * ldab + L) * 8u) | out);
        }
    };
    // ... and stores it at the position of its row, c - kv + t (lanes past
    // ldab write zeros at positions no band row of the column has)
    auto commit = [&](int k) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kChunk; ++q) {
            const int c = k * kChunk + q;
            ring[(c & 63) * 64 + ((c - kv + L) & 63)] = stg[q];
        }
    };
    // columns q0, q0+1 of chunk k, for the backward steps, which spread a
    // chunk's loads and ring stores over 16 steps each
    auto stage2 = [&]<int q0>(int k) __attribute__((always_inline)) {
#pragma unroll
        for (int q = q0; q < q0 + 2; ++q) {
            const int c = k * kChunk + q;
            const uint32_t out = lane_out | (((k >= 0) & (c < n)) ? 0u : kOutside);
            stg[q] = buf_ld(ab, (uint32_t(c * ldab + L) * 8u) | out);
        }
    };
    auto commit2 = [&]<int q0>(int k) __attribute__((always_inline)) {
#pragma unroll
        for (int q = q0; q < q0 + 2; ++q) {
            const int c = k * kChunk + q;
            ring[(c & 63) * 64 + ((c - kv + L) & 63)] = stg[q];
        }
    };
    auto ldb_ = [&](int r) { return buf_ld(bb, (r >= 0 && r < n) ? uint32_t(r) * 8u : kOutside); };
    auto stb_ = [&](int r, double v) { buf_st(bb, (r >= 0 && r < n) ? uint32_t(r) * 8u : kOutside, v); };

    // ------------------------------------------------------------ forward --
    if (kl > 0 && n > 1) {
        // at step j lane L holds row j + ((L - j) & 63)
        double b = ldb_(L), bn1 = ldb_(64 + L), bn2 = ldb_(128 + L);
        int myrow = L;
        int ipv = buf_ld_i32(pb, L < n ? uint32_t(L) * 4u : kOutside);
        int ipvn = buf_ld_i32(pb, 64 + L < n ? uint32_t(64 + L) * 4u : kOutside);
        double yfin = 0.0;
        double bnx;  // b rows and interchanges two blocks ahead, loaded early in a block
        int ipx;
        stage(0);
        commit(0);
        const unsigned long long act0 = lane_low(kl) << 1;  // rows j+1..j+kl
        double lr[8];  // this lane's multipliers, by step mod 8, read 4-5 steps ahead
#pragma unroll
        for (int q = 0; q < 4; ++q) lr[q] = ring[q * 64 + L];
        // the last step's update as formed, before the select keeps it in
        // the lanes that take part: the lane of row j always does, so b(j)
        // can be read there, one instruction earlier on the chain
        double t = b;
        // SWP: the block has interchanges (a copy without the test runs the
        // blocks that have none)
        auto fstep = [&]<bool EDGE, bool SWP, int Q>(int j, unsigned long long swp)
                         __attribute__((always_inline)) {
            if (!(EDGE && j >= n - 1)) {
                if (SWP && ((swp >> Q) & 1ull)) {
                    // the interchange of ipiv[j]: rows j and ipiv[j]-1 exchange values
                    const int lp = (__builtin_amdgcn_readlane(ipv, Q) - 1) & 63;
                    const double vq = readlane_d(b, Q), vp = readlane_d(b, lp);
                    b = __builtin_amdgcn_inverse_ballot_w64(lane_bit(Q)) ? vp
                                                                     : (lane_opaque_v(L) == lp ? vq : b);
                }
                const double bj = readlane_d((EDGE || SWP) ? b : t, Q);
                const double l = lr[Q & 7];
                if constexpr ((Q & 1) == 0) {
                    // two steps' multipliers, one slot apart: one LDS read
                    lr[(Q + 4) & 7] = ring[((Q + 4) & 63) * 64 + L];
                    lr[(Q + 5) & 7] = ring[((Q + 5) & 63) * 64 + L];
                }
                // chunk k+1 is loaded at the first step of chunk k and enters
                // the ring 27 steps later, before step 32k+28 reads its first
                // column: no staged register lives across the end of a block,
                // where the copies of the block join (a join would wait there
                // for every load in flight). Spread over the steps as in the
                // backward pass, the loads and stores measured slower here:
                // this chain has fewer idle issue slots to hide them in.
                if constexpr (Q == 0 || Q == 32) stage((j >> 5) + 1);
                if constexpr (Q == 27 || Q == 59) commit((j >> 5) + 1);
                t = __builtin_fma(-l, bj, b);
                if (EDGE) {
                    unsigned long long act = lane_mask(act0, Q);
                    act &= __builtin_amdgcn_ballot_w64(j + ((lane_opaque_v(L) - Q) & 63) < n);
                    if (__builtin_amdgcn_inverse_ballot_w64(act)) b = t;
                } else if (((lane_opaque_v(L) - Q - 1) & 63) < kl) {
                    // rows j+1..j+kl, by a vector compare: a select on a lane
                    // mask made by scalar instructions waits longer for it
                    b = t;
                }
                if (!BULK && __builtin_amdgcn_inverse_ballot_w64(lane_bit(Q))) {  // the lane of row j
                    yfin = bj;
                    b = bn1;
                }
            }
            if constexpr (Q == 1) {
                const int j0 = j - 1;
                bnx = ldb_(j0 + 192 + L);
                ipx = buf_ld_i32(pb, j0 + 128 + L < n ? uint32_t(j0 + 128 + L) * 4u : kOutside);
            }
            if constexpr (BULK && (Q == 31 || Q == 63)) {
                // lanes Q-31..Q have had their pivot steps: their rows are final
                if (__builtin_amdgcn_inverse_ballot_w64(Q == 31 ? lane_below(32) : ~lane_below(32))) {
                    stb_(myrow, b);
                    myrow += 64;
                    b = bn1;
                }
            }
        };
        for (int j0 = 0; j0 < (BULK ? n - 1 : n); j0 += 64) {
            // steps of this block that interchange
            const unsigned long long swp =
                __builtin_amdgcn_ballot_w64(j0 + L < n - 1 && ipv != j0 + L + 1);
            const bool edge = j0 + 64 >= n - 1;
            [&]<int... Qs>(std::integer_sequence<int, Qs...>) __attribute__((always_inline)) {
                if (edge)
                    (fstep.template operator()<true, true, Qs>(j0 + Qs, swp), ...);
                else if (swp != 0)
                    (fstep.template operator()<false, true, Qs>(j0 + Qs, swp), ...);
                else
                    (fstep.template operator()<false, false, Qs>(j0 + Qs, swp), ...);
            }(std::make_integer_sequence<int, 64>{});
            if (!BULK) {
                // rows j0..j0+63 are final (row n-1, never a pivot, is in b)
                const int r = j0 + L;
                stb_(r, r == n - 1 ? b : yfin);
            }
            bn1 = bn2;
            bn2 = bnx;
            ipv = ipvn;
            ipvn = ipx;
        }
        if (BULK) stb_(myrow, b);  // the rows no batch has stored
        // the backward pass reads these stores back
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "agent");
    }

    // ----------------------------------------------------------- backward --
    {
        const int top = n - 1;
        const int jt = top & ~63;
        // at step j lane L holds row j - ((j - L) & 63)
        int myrow = top - ((top - L) & 63);
        double b = ldb_(myrow);
        double bn1 = ldb_(jt - 64 + L), bn2 = ldb_(jt - 128 + L);
        double xfin = 0.0;
        double bnx;  // b rows two blocks ahead, loaded early in a block
        // chunk k-1 is loaded over the top 16 steps of chunk k (columns 2p,
        // 2p+1 at j = 32k+31-p; a burst of 32 loads, or of 32 ring stores,
        // holds up the step chain behind it) and each pair enters the ring
        // 12 steps later, by j = 32k+4, before step 32k+1 reads the chunk's
        // last column. No staged register lives across the end of a block.
        // Chunk kt-1 is also loaded and stored here whole: the steps above
        // the top row that would load part of it do not run (the pairs the
        // loop loads again are the same values).
        const int kt = top >> 5;
        stage(kt);
        commit(kt);
        stage(kt - 1);
        commit(kt - 1);
        // rows j-kv..j-1, relative to the lane of row j
        const unsigned long long act0 = kv == 0 ? 0ull : lane_low(kv) << (64 - kv);
        // this lane's u(i,j) and u(j,j) by step mod 4, read 2-3 steps ahead
        // (two steps at a time, at odd steps); steps top..top-2 read here,
        // placed by value selects (a slot index known only at run time would
        // put the arrays in scratch memory)
        double ur[4] = {}, dr[4] = {};
        {
#pragma unroll
            for (int d = 0; d < 3; ++d) {
                const int q = (top - d) & 63;
                const double uv = ring[q * 64 + L], dv = ring[q * 65];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    ur[i] = (q & 3) == i ? uv : ur[i];
                    dr[i] = (q & 3) == i ? dv : dr[i];
                }
            }
        }
        double t = b;  // as in the forward pass: the last step's update as formed
        auto bstep = [&]<bool EDGE, int Q>(int j) __attribute__((always_inline)) {
            if (!(EDGE && j > top)) {
                const double bj = readlane_d(EDGE ? b : t, Q);
                const double x = bj / dr[Q & 3];
                const double u = ur[Q & 3];
                if constexpr (Q & 1) {
                    // steps j-2 and j-3, one slot apart: one LDS read each for
                    // the lane's entries and for the diagonal (row j-2 sits at
                    // position Q2)
                    constexpr int Q2 = (Q - 2) & 63, Q3 = (Q - 3) & 63;
                    ur[Q2 & 3] = ring[Q2 * 64 + L];
                    ur[Q3 & 3] = ring[Q3 * 64 + L];
                    dr[Q2 & 3] = ring[Q2 * 65];
                    dr[Q3 & 3] = ring[Q3 * 65];
                }
                constexpr int Qh = Q & 31;
                if constexpr (Qh >= 16) stage2.template operator()<2 * (31 - Qh)>((j >> 5) - 1);
                if constexpr (Qh >= 4 && Qh < 20) commit2.template operator()<2 * (19 - Qh)>((j >> 5) - 1);
                t = __builtin_fma(-u, x, b);
                if (EDGE) {
                    unsigned long long act = lane_mask(act0, Q);
                    act &= __builtin_amdgcn_ballot_w64(j - ((Q - lane_opaque_v(L)) & 63) >= 0);
                    if (__builtin_amdgcn_inverse_ballot_w64(act)) b = t;
                } else if (((Q - lane_opaque_v(L) - 1) & 63) < kv) {
                    b = t;  // rows j-kv..j-1
                }
                if (__builtin_amdgcn_inverse_ballot_w64(lane_bit(Q))) {  // the lane of row j
                    xfin = x;
                    if (!BULK) b = bn1;
                }
            }
            if constexpr (Q == 62) bnx = ldb_(j - 62 - 192 + L);
            if constexpr (BULK && (Q == 32 || Q == 0)) {
                // lanes Q..Q+31 have had their pivot steps, except in the first
                // block those whose row is already below it
                if (__builtin_amdgcn_inverse_ballot_w64(Q == 32 ? ~lane_below(32) : lane_below(32)) &&
                    myrow >= j - Q) {
                    if (myrow <= top) stb_(myrow, xfin);
                    myrow -= 64;
                    b = bn1;
                }
            }
        };
        for (int j0 = jt; j0 >= 0; j0 -= 64) {
            // (with no superdiagonals no lane takes part in a step, and b(j)
            // is read from b)
            const bool edge = j0 + 63 > top || j0 == 0 || kv == 0;
            [&]<int... Qs>(std::integer_sequence<int, Qs...>) __attribute__((always_inline)) {
                if (edge)
                    (bstep.template operator()<true, 63 - Qs>(j0 + 63 - Qs), ...);
                else
                    (bstep.template operator()<false, 63 - Qs>(j0 + 63 - Qs), ...);
            }(std::make_integer_sequence<int, 64>{});
            if (!BULK) {
                const int r = j0 + L;
                if (r <= top) stb_(r, xfin);
            }
            bn1 = bn2;
            bn2 = bnx;
        }
    }
}

}  // namespace

bool getrs_lane_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab) {
    return kl + ku <= 63 && ldab <= 64 && ldab * n * 8 <= kMaxBufferBytes && n * 8 <= kMaxBufferBytes;
}

int launch_getrs_lane(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    if (!getrs_lane_fits(n, kl, ku, ldab)) {
        set_error("band_getrs: the lane solve needs kl+ku <= 63 and ldab <= 64");
        return BANDLU_ERR_UNSUPPORTED;
    }
    LaneParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.B = dB;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    P.ldb = ldb;
    P.strideB = strideB;
    P.n = (int)n;
    P.kl = (int)kl;
    P.kv = (int)(kl + ku);
    P.nrhs = (int)nrhs;
    if (kl + ku <= 32)
        hipLaunchKernelGGL(getrs_lane_kernel<true>, dim3((unsigned)(batch * nrhs)), dim3(64), 0, s, P);
    else
        hipLaunchKernelGGL(getrs_lane_kernel<false>, dim3((unsigned)(batch * nrhs)), dim3(64), 0, s, P);
    BANDLU_CHECK_LAUNCH("band_getrs (lane per row)");
    return BANDLU_OK;
}

}  // namespace bandlu
