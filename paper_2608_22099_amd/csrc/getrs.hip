// Solve with the band factors (xGBTRS, no transpose): the "lu(A) \ B" that
// Listings 1 and 2 end with.
//
// One wavefront solves one right-hand side of one system.  The right-hand
// side lives in LDS when it fits (else it is updated in place in global
// memory); lane t applies the update of row j+t (forward, t = 1..kl) or row
// j-t (backward, t = 1..kl+ku).  The factor column each step needs is loaded
// D steps ahead into a register ring, so the step chain never waits on HBM.
#include <algorithm>

#include "bufio.hpp"
#include "common.hpp"

#include <utility>

namespace bandlu {

int launch_getrs_ring(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s);
bool getrs_ring_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab);
int launch_getrs_lane(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s);
bool getrs_lane_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab);

namespace {

struct RsParams {
    const double *AB;
    const int32_t *ipiv;
    double *B;
    int64_t n, kl, ku, nrhs, ldab, strideAB, strideP, ldb, strideB;
};

constexpr int64_t kLdsMaxN = 8192;  // 64 KiB of LDS per right-hand side


template <int W, int D, bool LDS>
__global__ __launch_bounds__(64) void getrs_kernel(RsParams P) {
    extern __shared__ double smem[];
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    const int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    double *Bg = P.B + b * P.strideB + k * P.ldb;
    double *x = LDS ? smem : Bg;
    const int lane = threadIdx.x;
    const int64_t n = P.n, kl = P.kl, kv = P.kl + P.ku, ldab = P.ldab;
    if (LDS) {
        for (int64_t i = lane; i < n; i += 64) x[i] = Bg[i];
        __syncthreads();
    }
    // forward: L with the row interchanges
    if (kl > 0 && n > 1) {
        auto lfetch = [&](int64_t j, int w) -> double {
            const int64_t t = 1 + lane + 64 * w;
            return (j < n - 1 && t <= min(kl, n - 1 - j)) ? AB[j * ldab + kv + t] : 0.0;
        };
        double lr[D][W];
        int ip[D];
#pragma unroll
        for (int u = 0; u < D; ++u) {
#pragma unroll
            for (int w = 0; w < W; ++w) lr[u][w] = lfetch(u, w);
            ip[u] = u < n - 1 ? ipiv[u] : 0;
        }
        for (int64_t j0 = 0; j0 < n - 1; j0 += D) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int64_t j = j0 + u;
                        if (j >= n - 1) return;
                        int64_t l = ip[u] - 1;
                        if (l < j || l >= n) l = j;  // never touch memory off the vector
                        if (lane == 0 && l != j) {
                            const double t = x[l];
                            x[l] = x[j];
                            x[j] = t;
                        }
                        __syncthreads();
                        const double bj = x[j];
                        const int64_t km = min(kl, n - 1 - j);
#pragma unroll
                        for (int w = 0; w < W; ++w) {
                            const int64_t t = 1 + lane + 64 * w;
                            if (t <= km) x[j + t] = __builtin_fma(-lr[u][w], bj, x[j + t]);
                        }
                        __syncthreads();
#pragma unroll
                        for (int w = 0; w < W; ++w) lr[u][w] = lfetch(j + D, w);
                        ip[u] = j + D < n - 1 ? ipiv[j + D] : 0;
                    }(),
                    ...);
            }(std::make_integer_sequence<int, D>{});
        }
    }
    // backward: U with kl+ku superdiagonals
    {
        auto ufetch = [&](int64_t j, int w) -> double {
            const int64_t t = lane + 64 * w;
            return (j >= 0 && t <= min(kv, j)) ? AB[j * ldab + kv - t] : 0.0;
        };
        double ur[D][W];
#pragma unroll
        for (int u = 0; u < D; ++u)
#pragma unroll
            for (int w = 0; w < W; ++w) ur[u][w] = ufetch(n - 1 - u, w);
        for (int64_t j0 = n - 1; j0 >= 0; j0 -= D) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int64_t j = j0 - u;
                        if (j < 0) return;
                        if (lane == 0) x[j] = x[j] / ur[u][0];
                        __syncthreads();
                        const double bj = x[j];
                        const int64_t tm = min(kv, j);
#pragma unroll
                        for (int w = 0; w < W; ++w) {
                            const int64_t t = lane + 64 * w;
                            if (t >= 1 && t <= tm) x[j - t] = __builtin_fma(-ur[u][w], bj, x[j - t]);
                        }
                        __syncthreads();
#pragma unroll
                        for (int w = 0; w < W; ++w) ur[u][w] = ufetch(j - D, w);
                    }(),
                    ...);
            }(std::make_integer_sequence<int, D>{});
        }
    }
    if (LDS) {
        for (int64_t i = lane; i < n; i += 64) Bg[i] = x[i];
    }
}

// Register-window solve for narrow bands (kl <= 63, kl + ku < 64 * CPL), one
// wavefront per right-hand side.  Each step costs a few instructions: the
// right-hand side row the step finishes is read from its lane, and the rows
// it updates apply one fused multiply-add under a lane mask that the scalar
// unit rotates by one lane per step.
//
// Forward: row r lives in lane r mod 64.  Step j reads b[j] from lane j mod 64
// (after the interchange with row ipiv[j]-1, an exchange between two lanes),
// lanes j+1..j+kl (mod 64) apply the multipliers of column j, lane j mod 64
// stores the finished row and takes row j+64.  Backward: row r lives in lane
// (n-1-r) mod 64, register slot ((n-1-r) / 64) mod CPL.  Step j divides the
// row by U(j,j), the rows j-kl-ku..j-1 apply the column of U, and the slot
// stores row j and takes row j - 64*CPL.  Columns of L and U are loaded 64
// steps ahead into a register ring, the rows that enter in one block of
// steps with one load; the step loop is unrolled by 64 * CPL so that every
// register index is a compile-time constant.

template <int START>
__device__ __forceinline__ unsigned long long rotl64(unsigned long long w) {
    constexpr int s = START & 63;
    if constexpr (s == 0) return w;
    else return (w << s) | (w >> (64 - s));
}

// lanes (START .. START+len-1) mod (64 * CPL) as CPL 64-bit words (len < 64 * CPL)
template <int CPL, int START>
__device__ __forceinline__ unsigned long long window_word(int len, int word) {
    if constexpr (CPL == 1) {
        const unsigned long long ones = len >= 64 ? ~0ull : ((1ull << len) - 1);
        return rotl64<START>(ones);
    } else {
        typedef unsigned __int128 u128;
        constexpr int s = START & 127;
        const u128 ones = (u128(1) << len) - 1;
        u128 w = ones;
        if constexpr (s != 0) w = (ones << s) | (ones >> (128 - s));
        return (unsigned long long)(word == 0 ? w : (w >> 64));
    }
}

template <int CPL>
__global__ __launch_bounds__(64) void getrs_win_kernel(RsParams P) {
    constexpr int M = 64 * CPL;
    constexpr int DB = 64 / CPL;  // backward ring depth per slot
    const int L = threadIdx.x;
    const int64_t sys = blockIdx.x;
    const int64_t bidx = sys / P.nrhs, k = sys - bidx * P.nrhs;
    const int n = int(P.n), kl = int(P.kl), kv = int(P.kl + P.ku), ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + bidx * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    const Buf pb = make_buf(P.ipiv + bidx * P.strideP, uint32_t(int64_t(n) * 4));
    const Buf xb = make_buf(P.B + bidx * P.strideB + k * P.ldb, uint32_t(int64_t(n) * 8));
    auto rowoff = [](int r) -> uint32_t { return uint32_t(r) * 8u; };  // r < 0 or r >= n: outside

    // ------------------------------------------------------------ forward --
    if (kl > 0 && n > 1) {
        double bv = buf_ld(xb, rowoff(L));
        double nxt = buf_ld(xb, rowoff(64 + L));
        int ipv = buf_ld_i32(pb, uint32_t(L) * 4u);
        double lr[64];
        // the multiplier of column j for the row in lane L sits kv + ((L - j) mod 64)
        // entries into column j (the lanes outside the window read values they ignore)
        // (the column base, or an offset past every buffer, is chosen on the scalar
        // unit and added to the lane's part: the whole offset is range-checked)
        auto loff = [&](int u, int j) -> uint32_t {
            return uint32_t(kv + ((L - u) & 63)) * 8u + (j < n ? uint32_t(j * ldab) * 8u : kOutside);
        };
#pragma unroll
        for (int u = 0; u < 64; ++u) lr[u] = buf_ld(ab, loff(u, u));
        for (int j0 = 0; j0 < n - 1; j0 += 64) {
            const int ipv_next = buf_ld_i32(pb, uint32_t(j0 + 64 + L) * 4u);
            const double nxt_next = buf_ld(xb, rowoff(j0 + 128 + L));
            double done = 0.0;  // lane u: row j0 + u once step j0 + u has made it final
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int j = j0 + u;
                        if (j >= n - 1) return;
                        const int p = __builtin_amdgcn_readlane(ipv, u) - 1;
                        if (unsigned(p - j - 1) < unsigned(min(kl, n - 1 - j))) {
                            const int ls = p & 63;
                            const double vj = readlane_d(bv, u);
                            const double vp = readlane_d(bv, ls);
                            bv = L == u ? vp : (L == ls ? vj : bv);
                        }
                        const double bj = readlane_d(bv, u);
                        const int km = min(kl, n - 1 - j);
                        if (__builtin_amdgcn_inverse_ballot_w64(window_word<1, u + 1>(km, 0)))
                            bv = __builtin_fma(-lr[u], bj, bv);
                        if (__builtin_amdgcn_inverse_ballot_w64(1ull << u)) {
                            done = bv;  // row j is final
                            bv = nxt;   // row j + 64 enters
                        }
                        lr[u] = buf_ld(ab, loff(u, j + 64));
                    }(),
                    ...);
            }(std::make_integer_sequence<int, 64>{});
            // rows j0 .. j0+63 that are final (row n-1 is stored after the loop)
            buf_st(xb, j0 + L < n - 1 ? rowoff(j0 + L) : kOutside, done);
            ipv = ipv_next;
            nxt = nxt_next;
        }
        buf_st(xb, L == ((n - 1) & 63) ? rowoff(n - 1) : kOutside, bv);
        __threadfence();
    }
    // ----------------------------------------------------------- backward --
    {
        // slot s of lane L holds row n-1 - (L + 64 s) - M*q for block q
        double bv[CPL], nxt[CPL];
#pragma unroll
        for (int s = 0; s < CPL; ++s) bv[s] = buf_ld(xb, rowoff(n - 1 - (L + 64 * s)));
        double ur[CPL][DB];
        // entry (j - t, j) of U, t = ((L + 64 s - m) mod M), sits kv - t entries into column j
        // (for lanes beyond the band kv - t is negative and the offset wraps to
        // some other entry of the range-checked buffer; those lanes are never used)
        auto uoff = [&](int s, int u, int j) -> uint32_t {
            return uint32_t(kv - ((L + 64 * s - u) & (M - 1))) * 8u +
                   (j >= 0 ? uint32_t(j * ldab) * 8u : kOutside);
        };
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int s = 0; s < CPL; ++s) ur[s][d] = buf_ld(ab, uoff(s, d, n - 1 - d));
        for (int m0 = 0; m0 < n; m0 += M) {
            double done[CPL];
#pragma unroll
            for (int s = 0; s < CPL; ++s) {
                nxt[s] = buf_ld(xb, rowoff(n - 1 - (m0 + M + L + 64 * s)));
                done[s] = 0.0;
            }
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        constexpr int lj = u & 63, sj = u >> 6;
                        const int j = n - 1 - (m0 + u);
                        if (j < 0) return;
                        const double z = bv[sj] / ur[sj][u % DB];
                        const double xj = readlane_d(z, lj);
                        const int tm = min(kv, j);
#pragma unroll
                        for (int s = 0; s < CPL; ++s) {
                            if (__builtin_amdgcn_inverse_ballot_w64(window_word<CPL, u + 1>(tm, s)))
                                bv[s] = __builtin_fma(-ur[s][u % DB], xj, bv[s]);
                        }
                        if (__builtin_amdgcn_inverse_ballot_w64(1ull << lj)) {
                            done[sj] = xj;       // row j is final
                            bv[sj] = nxt[sj];    // row j - M enters
                        }
#pragma unroll
                        for (int s = 0; s < CPL; ++s)
                            ur[s][u % DB] = buf_ld(ab, uoff(s, u + DB, j - DB));
                    }(),
                    ...);
            }(std::make_integer_sequence<int, M>{});
            // rows n-1-m0 .. n-M-m0 are final
#pragma unroll
            for (int s = 0; s < CPL; ++s) buf_st(xb, rowoff(n - 1 - (m0 + L + 64 * s)), done[s]);
        }
    }
}

// Batched solve for small bands (kl + ku <= 15): sixteen lanes per system,
// four systems per wavefront, all at the same step.  Row r of a right-hand
// side lives in lane r mod 16 of its group (forward) or lane (n-1-r) mod 16
// (backward); with the step loop unrolled by 16 the lane of the row a step
// finishes is a compile-time constant, so its value reaches the rest of the
// group by one DPP row broadcast.  The row interchange of the forward pass is
// a chain of selects over the group's pivot offset (skipped when no system
// of the wavefront pivots at that step).  One range-checked buffer per array
// spans the whole batch (the host checks that each is < 2 GiB).
template <int K>
__device__ __forceinline__ double rs_bcast(double v) {
    const long long x = __double_as_longlong(v);
    // (every lane is written: the old value is the source, no zeroing)
    const int lo = __builtin_amdgcn_update_dpp((int)(x & 0xffffffffll), (int)(x & 0xffffffffll),
                                               0x150 + K, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(x >> 32), (int)(x >> 32), 0x150 + K, 0xf, 0xf, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

template <int K>
__device__ __forceinline__ int rs_bcast_i(int v) {
    return __builtin_amdgcn_update_dpp(v, v, 0x150 + K, 0xf, 0xf, false);
}

// the 16-bit lane pattern `bits` (bit i = lane i of a group) in every group
__device__ __forceinline__ unsigned long long rs_groups(unsigned bits) {
    return 0x0001000100010001ull * (bits & 0xffffu);
}

// (kl is a template parameter: the interchange of the forward pass then
// tests exactly kl candidate rows, with no test of kl per candidate)
template <int KL>
__global__ __launch_bounds__(64) void getrs_g16_kernel(RsParams P, int64_t systems) {
    const int lane = threadIdx.x, gl = lane & 15;
    const int64_t sys = int64_t(blockIdx.x) * 4 + (lane >> 4);
    const bool live = sys < systems;
    const int64_t bidx = live ? sys / P.nrhs : 0, k = live ? sys - bidx * P.nrhs : 0;
    constexpr int kl = KL;
    const int n = int(P.n), kv = int(P.kl + P.ku), ldab = int(P.ldab);
    const int64_t batch = (systems + P.nrhs - 1) / P.nrhs;
    const Buf ab = make_buf(P.AB, uint32_t(batch * P.strideAB * 8));
    const Buf pb = make_buf(P.ipiv, uint32_t(batch * P.strideP * 4));
    const Buf xb = make_buf(P.B, uint32_t(batch * P.strideB * 8));
    const uint32_t abase = live ? uint32_t(bidx * P.strideAB * 8) : kOutside;
    const uint32_t pbase = live ? uint32_t(bidx * P.strideP * 4) : kOutside;
    const uint32_t xbase = live ? uint32_t((bidx * P.strideB + k * P.ldb) * 8) : kOutside;
    auto rowoff = [&](int r) -> uint32_t { return r >= 0 && r < n ? xbase + uint32_t(r) * 8u : kOutside; };

    // ------------------------------------------------------------ forward --
    if (KL > 0 && n > 1) {
        double bv = buf_ld(xb, rowoff(gl));
        double nxt = buf_ld(xb, rowoff(16 + gl));
        int ipv = buf_ld_i32(pb, gl < n ? pbase + uint32_t(gl) * 4u : kOutside);
        double lr[16];
        // multiplier of column j for the row in lane gl: kv + ((gl - j) mod 16) into column j
        auto loff = [&](int u, int j) -> uint32_t {
            return j < n ? abase + uint32_t(j * ldab + kv + ((gl - u) & 15)) * 8u : kOutside;
        };
#pragma unroll
        for (int u = 0; u < 16; ++u) lr[u] = buf_ld(ab, loff(u, u));
        // the multipliers' per-lane offsets for lean blocks (plus the scalar
        // (j + 16) * ldab * 8)
        uint32_t ltab[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) ltab[u] = abase + uint32_t(kv + ((gl - u) & 15)) * 8u;
        // one step; LEAN: a block away from the end (kl rows below every
        // step, every load in range), where the update masks are constants
        auto fstep = [&]<int u, bool LEAN>(int j0, double &done) __attribute__((always_inline)) {
            const int j = j0 + u;
            if (!LEAN && j >= n - 1) return;
            const int km = LEAN ? KL : min(kl, n - 1 - j);
            const int toff = (gl - u) & 15;
            const int d = rs_bcast_i<u>(ipv) - 1 - j;  // pivot offset of this group
            if (__ballot(d != 0)) {
                // exchange rows j and j+d (0 < d <= km) inside each group
                const double bj0 = rs_bcast<u>(bv);
                double bjn = bj0;
                [&]<int... Ts>(std::integer_sequence<int, Ts...>) {
                    (
                        [&] {
                            constexpr int t = Ts + 1;
                            const double vt = rs_bcast<(u + t) & 15>(bv);
                            bjn = d == t ? vt : bjn;
                        }(),
                        ...);
                }(std::make_integer_sequence<int, KL>{});
                const bool ok = d > 0 && d <= km;
                bv = (ok && toff == 0) ? bjn : ((ok && toff == d) ? bj0 : bv);
            }
            const double bj = rs_bcast<u>(bv);
            if (__builtin_amdgcn_inverse_ballot_w64(rs_groups(((1u << km) - 1) << (u + 1) |
                                                              ((1u << km) - 1) >> (15 - u))))
                bv = __builtin_fma(-lr[u], bj, bv);
            if (__builtin_amdgcn_inverse_ballot_w64(rs_groups(1u << u))) {
                done = bv;  // row j is final
                bv = nxt;   // row j + 16 enters
            }
            if constexpr (LEAN)
                lr[u] = buf_ld_so(ab, ltab[u], uint32_t(j + 16) * uint32_t(ldab) * 8u);
            else
                lr[u] = buf_ld(ab, loff(u, j + 16));
        };
        auto fblock = [&]<bool LEAN>(int j0) __attribute__((always_inline)) {
            const int ipv_next =
                buf_ld_i32(pb, j0 + 16 + gl < n ? pbase + uint32_t(j0 + 16 + gl) * 4u : kOutside);
            const double nxt_next = buf_ld(xb, rowoff(j0 + 32 + gl));
            double done = 0.0;
            [&]<int... Us>(std::integer_sequence<int, Us...>) __attribute__((always_inline)) {
                (fstep.template operator()<Us, LEAN>(j0, done), ...);
            }(std::make_integer_sequence<int, 16>{});
            buf_st(xb, j0 + gl < n - 1 ? rowoff(j0 + gl) : kOutside, done);
            ipv = ipv_next;
            nxt = nxt_next;
        };
        // the lean blocks run in a loop of their own (no join with the other
        // block's code at the loop head, where every load in flight would be
        // waited for)
        auto flean = [&](int j0) { return j0 + 32 + KL <= n; };
        for (int j0 = 0; j0 < n - 1;) {
            if (flean(j0)) {
                do {
                    fblock.template operator()<true>(j0);
                    j0 += 16;
                } while (flean(j0));
            } else {
                fblock.template operator()<false>(j0);
                j0 += 16;
            }
        }
        buf_st(xb, gl == ((n - 1) & 15) ? rowoff(n - 1) : kOutside, bv);
        __threadfence();
    }
    // ----------------------------------------------------------- backward --
    {
        double bv = buf_ld(xb, rowoff(n - 1 - gl));
        double ur[16];
        // entry (j - t, j) of U, t = (gl - m) mod 16, sits kv - t entries into column j
        auto uoff = [&](int u, int j) -> uint32_t {
            return j >= 0 ? abase + uint32_t(j * ldab + kv - ((gl - u) & 15)) * 8u : kOutside;
        };
#pragma unroll
        for (int u = 0; u < 16; ++u) ur[u] = buf_ld(ab, uoff(u, n - 1 - u));
        // the U entries' per-lane offsets for lean blocks (plus the scalar
        // (j - 32) * ldab * 8; lean blocks have j >= 32, and every per-lane
        // part is positive)
        uint32_t utab[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) utab[u] = abase + uint32_t(16 * ldab + kv - ((gl - u) & 15)) * 8u;
        // one step; LEAN: a block with kv rows above every step and every
        // load in range (the update masks then do not change from block to
        // block)
        auto bstep = [&]<int u, bool LEAN>(int m0, double &done, double nxt) __attribute__((always_inline)) {
            const int j = n - 1 - (m0 + u);
            if (!LEAN && j < 0) return;
            const double xj = rs_bcast<u>(bv / ur[u]);
            const int tm = LEAN ? kv : min(kv, j);
            if (__builtin_amdgcn_inverse_ballot_w64(rs_groups(((1u << tm) - 1) << (u + 1) |
                                                              ((1u << tm) - 1) >> (15 - u))))
                bv = __builtin_fma(-ur[u], xj, bv);
            if (__builtin_amdgcn_inverse_ballot_w64(rs_groups(1u << u))) {
                done = xj;  // row j is final
                bv = nxt;   // row j - 16 enters
            }
            if constexpr (LEAN)
                ur[u] = buf_ld_so(ab, utab[u], uint32_t(j - 32) * uint32_t(ldab) * 8u);
            else
                ur[u] = buf_ld(ab, uoff(u, j - 16));
        };
        auto bblock = [&]<bool LEAN>(int m0) __attribute__((always_inline)) {
            const double nxt = buf_ld(xb, rowoff(n - 1 - (m0 + 16 + gl)));
            double done = 0.0;
            [&]<int... Us>(std::integer_sequence<int, Us...>) __attribute__((always_inline)) {
                (bstep.template operator()<Us, LEAN>(m0, done, nxt), ...);
            }(std::make_integer_sequence<int, 16>{});
            buf_st(xb, rowoff(n - 1 - (m0 + gl)), done);
        };
        // lean: every step of the block has j >= max(32, kv); the lean blocks
        // run in a loop of their own, as in the forward pass
        auto blean = [&](int m0) { return m0 + 48 + kv <= n; };
        for (int m0 = 0; m0 < n;) {
            if (blean(m0)) {
                do {
                    bblock.template operator()<true>(m0);
                    m0 += 16;
                } while (blean(m0));
            } else {
                bblock.template operator()<false>(m0);
                m0 += 16;
            }
        }
    }
}

// Any band: one workgroup of 256 threads per right-hand side, the vector in
// LDS when it fits (else updated in place in global memory), two barriers per
// step.  Each entry receives its fused multiply-adds in the order of the
// sequence above, so the result is bitwise that of the narrower kernels.
constexpr int kAnyThreads = 256;

template <bool LDS>
__global__ __launch_bounds__(kAnyThreads) void getrs_any_kernel(RsParams P) {
    extern __shared__ double smem[];
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    const int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    double *Bg = P.B + b * P.strideB + k * P.ldb;
    double *x = LDS ? smem : Bg;
    const int tid = threadIdx.x;
    const int64_t n = P.n, kl = P.kl, kv = P.kl + P.ku, ldab = P.ldab;
    if (LDS) {
        for (int64_t i = tid; i < n; i += kAnyThreads) x[i] = Bg[i];
    }
    __syncthreads();
    if (kl > 0) {
        for (int64_t j = 0; j < n - 1; ++j) {
            const int64_t km = min(kl, n - 1 - j);
            if (tid == 0) {
                const int64_t l = ipiv[j] - 1;
                if (l != j && l > j && l < n) {
                    const double t0 = x[l];
                    x[l] = x[j];
                    x[j] = t0;
                }
            }
            __syncthreads();
            const double xj = x[j];
            const double *lc = AB + j * ldab + kv;
            for (int64_t t = 1 + tid; t <= km; t += kAnyThreads)
                x[j + t] = __builtin_fma(-lc[t], xj, x[j + t]);
            __syncthreads();
        }
    }
    for (int64_t j = n - 1; j >= 0; --j) {
        const double *uc = AB + j * ldab + kv - j;  // uc[i] = U(i, j)
        if (tid == 0) x[j] = x[j] / uc[j];
        __syncthreads();
        const double xj = x[j];
        for (int64_t i = max(int64_t(0), j - kv) + tid; i < j; i += kAnyThreads)
            x[i] = __builtin_fma(-uc[i], xj, x[i]);
        __syncthreads();
    }
    if (LDS) {
        for (int64_t i = tid; i < n; i += kAnyThreads) Bg[i] = x[i];
    }
}

template <int W>
constexpr int rs_depth() { return W >= 16 ? 2 : 32 / W; }

template <int W>
int launch_w(bool lds, const RsParams &P, int64_t systems, hipStream_t s) {
    constexpr int D = rs_depth<W>();
    if (lds) {
        hipLaunchKernelGGL((getrs_kernel<W, D, true>), dim3((unsigned)systems), dim3(64),
                           size_t(P.n) * sizeof(double), s, P);
    } else {
        hipLaunchKernelGGL((getrs_kernel<W, D, false>), dim3((unsigned)systems), dim3(64), 0, s,
                           P);
    }
    BANDLU_CHECK_LAUNCH("band_getrs");
    return BANDLU_OK;
}

bool g16_fits(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, int64_t strideAB, int64_t strideP,
              int64_t ldb, int64_t strideB, int64_t batch) {
    return kl + ku <= 15 && batch * strideAB * 8 <= kMaxBufferBytes &&
           batch * strideP * 4 <= kMaxBufferBytes && batch * strideB * 8 <= kMaxBufferBytes &&
           ldb * nrhs <= strideB;
}

bool window_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab) {
    return ldab * n * 8 <= kMaxBufferBytes && n * 8 <= kMaxBufferBytes && kl <= 63 && kl + ku < 128;
}

int select_getrs(int64_t n, int64_t kl, int64_t ku, int64_t ldab, int64_t nrhs, int64_t strideAB,
                 int64_t strideP, int64_t ldb, int64_t strideB, int64_t batch) {
    const int64_t systems = batch * nrhs;
    if (systems >= 64 && g16_fits(n, kl, ku, nrhs, strideAB, strideP, ldb, strideB, batch))
        return BANDLU_GETRS_G16;
    if (getrs_lane_fits(n, kl, ku, ldab)) return BANDLU_GETRS_LANE;
    if (getrs_ring_fits(n, kl, ku, ldab)) return BANDLU_GETRS_RING;
    if (window_fits(n, kl, ku, ldab)) return BANDLU_GETRS_WINDOW;
    return BANDLU_GETRS_GENERIC;
}

int launch_getrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                 int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                 double *dB, int64_t ldb, int64_t strideB, int64_t batch, int variant,
                 hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    RsParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.B = dB;
    P.n = n;
    P.kl = kl;
    P.ku = ku;
    P.nrhs = nrhs;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    P.ldb = ldb;
    P.strideB = strideB;
    const int64_t systems = batch * nrhs;
    if (systems > INT32_MAX) {
        set_error("band_getrs: batch * nrhs too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    int v = variant;
    if (v == 0) {
        v = select_getrs(n, kl, ku, ldab, nrhs, strideAB, strideP, ldb, strideB, batch);
    } else {
        const bool ok = v == BANDLU_GETRS_G16 ? g16_fits(n, kl, ku, nrhs, strideAB, strideP, ldb, strideB, batch)
                      : v == BANDLU_GETRS_RING ? getrs_ring_fits(n, kl, ku, ldab)
                      : v == BANDLU_GETRS_WINDOW ? window_fits(n, kl, ku, ldab)
                      : v == BANDLU_GETRS_LANE ? getrs_lane_fits(n, kl, ku, ldab)
                      : v == BANDLU_GETRS_GENERIC;
        if (!ok) {
            set_error("band_getrs: variant %d cannot solve n = %lld, kl = %lld, ku = %lld", v,
                      (long long)n, (long long)kl, (long long)ku);
            return BANDLU_ERR_UNSUPPORTED;
        }
    }
    // many systems with a small band: sixteen lanes per system
    if (v == BANDLU_GETRS_G16) {
        using G16 = void (*)(RsParams, int64_t);
        static constexpr G16 g16[16] = {
            getrs_g16_kernel<0>,  getrs_g16_kernel<1>,  getrs_g16_kernel<2>,  getrs_g16_kernel<3>,
            getrs_g16_kernel<4>,  getrs_g16_kernel<5>,  getrs_g16_kernel<6>,  getrs_g16_kernel<7>,
            getrs_g16_kernel<8>,  getrs_g16_kernel<9>,  getrs_g16_kernel<10>, getrs_g16_kernel<11>,
            getrs_g16_kernel<12>, getrs_g16_kernel<13>, getrs_g16_kernel<14>, getrs_g16_kernel<15>};
        // (g16_fits: kl + ku <= 15)
        hipLaunchKernelGGL(g16[kl], dim3((unsigned)((systems + 3) / 4)), dim3(64), 0, s, P,
                           systems);
        BANDLU_CHECK_LAUNCH("band_getrs (16 lanes per system)");
        return BANDLU_OK;
    }
    if (v == BANDLU_GETRS_LANE)
        return launch_getrs_lane(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb,
                                 strideB, batch, s);
    if (v == BANDLU_GETRS_RING)
        return launch_getrs_ring(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb,
                                 strideB, batch, s);
    if (v == BANDLU_GETRS_WINDOW) {
        if (kl + ku < 64) {
            hipLaunchKernelGGL(getrs_win_kernel<1>, dim3((unsigned)systems), dim3(64), 0, s, P);
        } else {
            hipLaunchKernelGGL(getrs_win_kernel<2>, dim3((unsigned)systems), dim3(64), 0, s, P);
        }
        BANDLU_CHECK_LAUNCH("band_getrs (window)");
        return BANDLU_OK;
    }
    const int64_t lanes_needed = std::max(kl, kl + ku + 1);
    const bool lds = n <= kLdsMaxN;
    if (lanes_needed <= 64) return launch_w<1>(lds, P, systems, s);
    if (lanes_needed <= 128) return launch_w<2>(lds, P, systems, s);
    if (lanes_needed <= 256) return launch_w<4>(lds, P, systems, s);
    if (lanes_needed <= 512) return launch_w<8>(lds, P, systems, s);
    if (lanes_needed <= 1024) return launch_w<16>(lds, P, systems, s);
    if (lds) {
        hipLaunchKernelGGL(getrs_any_kernel<true>, dim3((unsigned)systems), dim3(kAnyThreads),
                           size_t(n) * sizeof(double), s, P);
    } else {
        hipLaunchKernelGGL(getrs_any_kernel<false>, dim3((unsigned)systems), dim3(kAnyThreads), 0,
                           s, P);
    }
    BANDLU_CHECK_LAUNCH("band_getrs (any band)");
    return BANDLU_OK;
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int band_getrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                          int64_t ldab, const int32_t *d_ipiv, double *dB, int64_t ldb,
                          void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_getrs: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || d_ipiv != nullptr, 7, "band_getrs: d_ipiv is null");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 8, "band_getrs: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 9, "band_getrs: ldb < max(1, n)");
    if (n > kMaxN) {
        set_error("band_getrs: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrs(n, kl, ku, nrhs, dAB, ldab, ldab * n, d_ipiv, n, dB, ldb, ldb * nrhs, 1, 0,
                        as_stream(stream));
}

extern "C" int band_getrs_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs,
                                  const double *dAB, int64_t ldab, int64_t strideAB,
                                  const int32_t *d_ipiv, int64_t strideP, double *dB,
                                  int64_t ldb, int64_t strideB, int64_t batch, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs_batched: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs_batched: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_getrs_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_getrs_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 8, "band_getrs_batched: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 9, "band_getrs_batched: strideP < n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 10,
               "band_getrs_batched: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 11, "band_getrs_batched: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 12, "band_getrs_batched: strideB < ldb*nrhs");
    BANDLU_ARG(batch >= 0, 13, "band_getrs_batched: batch < 0");
    if (n > kMaxN) {
        set_error("band_getrs_batched: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrs(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb, strideB,
                        batch, 0, as_stream(stream));
}

extern "C" int band_getrs_ex(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                             int64_t ldab, int64_t strideAB, const int32_t *d_ipiv,
                             int64_t strideP, double *dB, int64_t ldb, int64_t strideB,
                             int64_t batch, int variant, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs_ex: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs_ex: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs_ex: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs_ex: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_getrs_ex: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs_ex: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_getrs_ex: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 8, "band_getrs_ex: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 9, "band_getrs_ex: strideP < n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 10, "band_getrs_ex: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 11, "band_getrs_ex: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 12, "band_getrs_ex: strideB < ldb*nrhs");
    BANDLU_ARG(batch >= 0, 13, "band_getrs_ex: batch < 0");
    BANDLU_ARG(variant >= 0 && variant <= BANDLU_GETRS_LANE, 14, "band_getrs_ex: unknown variant");
    if (n > kMaxN) {
        set_error("band_getrs_ex: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrs(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb, strideB,
                        batch, variant, as_stream(stream));
}

extern "C" int band_getrs_variant(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, int64_t batch) {
    const int64_t bmax = n > 1 ? n - 1 : 0;
    if (n < 0) return -1;
    if (kl < 0 || kl > bmax) return -2;
    if (ku < 0 || ku > bmax) return -3;
    if (nrhs < 0) return -4;
    if (batch < 0) return -5;
    const int64_t ldab = 2 * kl + ku + 1;
    const int64_t ldb = n > 1 ? n : 1;
    return select_getrs(n, kl, ku, ldab, nrhs, ldab * n, n, ldb, ldb * nrhs, batch);
}
