// Banded LU with partial pivoting (xGBTRF semantics), one matrix per
// wavefront, for 6 <= kl <= 31 and 2kl+ku+1 <= 64: the single-matrix kernel of
// Sec. III-A's specialised algorithm f(N) for narrow bands.
//
// Two layouts of the active window are kept side by side.
//   * Column c of the band window lives in lane c mod 64, its kl+1 window rows
//     in register slots (row mod H), H = kl + 1.  This copy takes the rank-1
//     updates, stores the finished rows of U and takes the rows that enter.
//   * The pivot column j and the next column j+1 are also held transposed:
//     row r in lane r mod 64 (registers y and z).  The pivot search is then a
//     wave-wide DPP maximum over y, the multipliers are formed in the lanes of
//     their rows, and column j+1 is brought up to date with one fused
//     multiply-add per lane, so the next step's pivot column (z) is ready as
//     soon as the multipliers are.  The column after that (j+2) is transposed
//     through LDS from its lane's window slots one step ahead, off the chain
//     of dependent pivot decisions.
// Lane predicates are 64-bit masks rotated on the scalar unit and applied as
// exec masks (no per-lane selects in the update), the reciprocal of every
// candidate is formed while the maximum is reduced, and the register slots
// are plain arrays indexed by compile-time constants (the step loop is
// unrolled by a multiple of H; a row interchange reaches its dynamic slot
// through a chain of selects on the wave-uniform pivot offset).  Every entry
// sees the same fused multiply-adds, in the same order, as in the unblocked
// algorithm.
#pragma once

#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"
#include "wave.hpp"

namespace bandlu {

// 64-bit masks on the scalar unit: `len` lanes starting at lane `start`,
// wrapping around (0 <= len <= 63).  The second shift is split so that no
// shift count reaches 64.
__device__ __forceinline__ unsigned long long lanes_from(int start, int len) {
    const unsigned long long ones = (1ull << len) - 1;
    const int s = start & 63;
    return (ones << s) | ((ones >> 1) >> (63 - s));
}

// rotate right by r (0 <= r <= 63): bit k of the result is bit r+k mod 64
__device__ __forceinline__ unsigned long long rotr64(unsigned long long m, int r) {
    return (m >> r) | ((m << 1) << (63 - r));
}

// Maximum over the 64 lanes of a 32-bit unsigned key, uniform: one DPP max per
// level inside rows of 16 lanes, then the four row maxima.
__device__ __forceinline__ unsigned wave_max_u32(unsigned v) {
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xf, 0xf, false));
    const unsigned a = max((unsigned)__builtin_amdgcn_readlane((int)v, 0), (unsigned)__builtin_amdgcn_readlane((int)v, 16));
    const unsigned b = max((unsigned)__builtin_amdgcn_readlane((int)v, 32), (unsigned)__builtin_amdgcn_readlane((int)v, 48));
    return max(a, b);
}

__device__ __forceinline__ bool in_mask(unsigned long long m) {
    return __builtin_amdgcn_inverse_ballot_w64(m);
}

template <int H, int PF>
__global__ __launch_bounds__(64) void getrf_win2_kernel(WinParams P) {
    static_assert(H >= 2 && H <= 32, "window of 2..32 rows");
    static_assert(PF % H == 0, "prefetch depth must be a multiple of H");
    constexpr int kl = H - 1;
    const int L = threadIdx.x;
    const int64_t b = blockIdx.x;  // one matrix per workgroup (= wavefront)
    const int n = P.n, ku = P.ku, kv = kl + P.ku, ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + b * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    const Buf pb = make_buf(P.ipiv + b * P.strideP, uint32_t(int64_t(n) * 4));
    __shared__ double s_col[64];  // column j+2, rows j+1..j+1+kl (every other slot)
    __shared__ double s_l[32];    // multipliers of column j by row offset

    // the column in [x, x+64) this lane holds
    auto colof = [&](int x) -> int { return x + ((L - x) & 63); };
    // original band entry (r, c), else outside
    auto foff = [&](int r, int c) -> uint32_t {
        const bool ok = c >= 0 && c < n && r >= 0 && r < n && unsigned(r - c + ku) <= unsigned(kl + ku);
        return ok ? uint32_t(c * ldab + kv + r - c) * 8u : kOutside;
    };

    double a[H];
    double pf[PF];
#pragma unroll
    for (int r = 0; r < H; ++r) a[r] = buf_ld(ab, foff(r, colof(r - H + 1)));
#pragma unroll
    for (int k = 0; k < PF; ++k) pf[k] = buf_ld(ab, foff(k + H, colof(k + 1)));
    // transposed columns 0 and 1 (rows 0..kl; lane = row)
    double y = buf_ld(ab, L <= kl ? foff(L, 0) : kOutside);
    double z = buf_ld(ab, L <= kl ? foff(L, 1) : kOutside);
    int ju = 0, info = 0;

    auto step = [&]<int U>(int j) __attribute__((always_inline)) {
        constexpr int S0 = U % H;
        if (j >= n) return;
        const int km = min(kl, n - 1 - j);
        const int u = j & 63;
        const int toff = (L - u) & 63;  // row offset of this lane in the transposed columns
        // ---- 1. pivot: first largest |y| over rows j..j+km.  The maximum is
        // taken over the high 32 bits of |y| (monotone in |y|); a NaN on the
        // diagonal ranks above everything, one below it ranks with the zeros
        // (so an earlier row always beats it).  Only when several rows tie on
        // the high word are the low words compared.
        const unsigned long long cand = lanes_from(u, km + 1);
        const double rall = 1.0 / y;  // every candidate's reciprocal, beside the reduction
        const bool nan = __builtin_isnan(y);
        const bool inc = in_mask(cand);
        const unsigned yhi = unsigned(__double_as_longlong(y) >> 32) & 0x7fffffffu;
        const unsigned khi = !inc ? 0u : (nan ? (toff == 0 ? 0x7ff00001u : 0u) : yhi);
        unsigned long long hit = __ballot(khi == wave_max_u32(khi)) & cand;
        if (__popcll(hit) > 1) {
            const bool tied = (hit >> L) & 1;
            const unsigned klo = (tied && !nan) ? unsigned(__double_as_longlong(y)) : 0u;
            hit &= __ballot(klo == wave_max_u32(klo));
        }
        const int p = __builtin_ctzll(rotr64(hit, u));  // first in row order
        const int lp = (u + p) & 63;
        const double piv = readlane_d(y, lp);
        // stores below: a wave-uniform offset inside the buffer on the scalar
        // unit plus the lane's part, which is an offset past every buffer for
        // the lanes that must not store
        buf_st_i32(pb, (L == 0 ? 0u : kOutside) + uint32_t(j) * 4u, j + p + 1);
        const uint32_t cbase = uint32_t(j * ldab + kv) * 8u;  // diagonal entry of column j
        const unsigned long long mrows = lanes_from(u + 1, km);  // rows j+1..j+km
        const uint32_t loff = in_mask(mrows) ? uint32_t(toff) * 8u : kOutside;
        if (piv != 0.0) {
            ju = max(ju, min(j + ku + p, n - 1));
            if (p != 0) {
                // ---- 2. interchange rows j and j+p
                const double y0 = readlane_d(y, u), z0 = readlane_d(z, u), zp = readlane_d(z, lp);
                y = L == u ? piv : (L == lp ? y0 : y);
                z = L == u ? zp : (L == lp ? z0 : z);
                if (in_mask(lanes_from(u, ju - j + 1))) win_swap<H, S0>(a, p);
            }
            // ---- 3. multipliers in the lanes of their rows
            double l;
            if (fabs(piv) >= DBL_MIN) {
                l = y * readlane_d(rall, lp);
            } else {
                l = y / piv;
            }
            buf_st_so(ab, loff, cbase, l);
            if (in_mask(mrows)) s_l[toff & 31] = l;
            // ---- 4. column j+1, transposed: ready for the next pivot search
            const double u1 = readlane_d(z, u);
            if (in_mask(mrows)) z = __builtin_fma(-l, u1, z);
        } else {
            // zero pivot: nothing is eliminated, the column below the diagonal stays
            if (info == 0) info = j + 1;
            buf_st_so(ab, loff, cbase, y);
        }
        // ---- 5. row j of U leaves the window, row j+H enters (before the
        // update below, which does not touch slot S0: this work hides the LDS
        // round trip of the multipliers)
        const double uu = a[S0];
        {
            // entry (j, j+t) of U sits at cbase + t (ldab-1), for lanes t = 0..kv
            const unsigned long long um = lanes_from(u, min(kv, n - 1 - j) + 1);
            buf_st_so(ab, in_mask(um) ? uint32_t(toff * (ldab - 1)) * 8u : kOutside, cbase, uu);
            a[S0] = pf[U];
            // step j+PF takes row r = c0 + kl of column c0 + t, c0 = j+PF+1, into the
            // lane holding that column: band entry iff t <= kv, at
            // (c0 ldab + kv + kl) + t (ldab-1)
            const int c0 = j + PF + 1;
            const int tn = (L - c0) & 63;
            const int len = c0 + kl < n ? min(kv, n - 1 - c0) + 1 : 0;
            const uint32_t rbase = uint32_t(c0 * ldab + kv + kl) * 8u;
            pf[U] = buf_ld_so(ab, in_mask(lanes_from(c0, len)) ? uint32_t(tn * (ldab - 1)) * 8u : kOutside,
                              c0 + kl < n ? rbase : 0u);
        }
        // ---- 6. next step's pivot column: z plus its entering row j+1+kl (now
        // in slot S0 of its lane)
        const double ent = readlane_d(a[S0], (j + 1) & 63);
        y = L == ((j + 1 + kl) & 63) ? ent : z;
        // ---- 7. rank-1 update of the window columns j+1..ju (near the end of the
        // matrix, multiplier slots t > km are stale: they only reach rows below
        // the matrix, which are never stored)
        if (piv != 0.0) {
            __builtin_amdgcn_wave_barrier();
            double lm[H];
#pragma unroll
            for (int t = 1; t < H; ++t) lm[t] = s_l[t];
            if (in_mask(lanes_from(u + 1, ju - j))) {
#pragma unroll
                for (int t = 1; t < H; ++t) a[(S0 + t) % H] = __builtin_fma(-lm[t], uu, a[(S0 + t) % H]);
            }
        }
        // ---- 8. column j+2 (updated) transposed through LDS for the next step
        if (L == ((j + 2) & 63)) {
            // every other slot: pairs of 64-bit stores take any two registers,
            // while a 128-bit store would need them copied next to each other
#pragma unroll
            for (int t = 0; t < H; ++t) s_col[2 * t] = a[(S0 + 1 + t) % H];
        }
        __builtin_amdgcn_wave_barrier();
        z = s_col[2 * (((L - u - 1) & 63) & 31)];
    };

    for (int j0 = 0; j0 < n; j0 += PF) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) {
            (step.template operator()<Us>(j0 + Us), ...);
        }(std::make_integer_sequence<int, PF>{});
    }
    if (L == 0) P.info[b] = info;
}

}  // namespace bandlu
