// Banded LU with partial pivoting (xGBTRF semantics), one matrix per
// wavefront, the active window in registers: the single-matrix kernel for
// narrow bands (Sec. III-A's specialised algorithm f(N)).
//
// Layout.  At step j the window is rows j..j+kl by columns j..j+kl+ku.  Column
// c lives in lane (c mod M) mod 64, register sub-slot (c mod M) / 64, with
// M = 64 * CPL >= 2kl+ku+1; row r of a column lives in element r mod H of a
// register vector (H = kl + 1).  The step loop is unrolled by PF, a multiple of
// H, so every element index except the pivot row's is a compile-time constant;
// the pivot row's index is wave-uniform and is reached with indexed register
// moves, never through scratch memory.
//
// Step j:
//   1. pivot search.  H <= 6: the lane holding column j scans its H values.
//      H > 6: that lane writes the column to LDS, lane t reads row j+t, and a
//      DPP max over the lanes plus a ballot gives the first index of the
//      largest magnitude (a NaN counts as largest in position 0 and smallest
//      elsewhere, which reproduces BLAS i_amax);
//   2. lanes whose column is in j..ju swap the elements of rows j and j+p;
//   3. multipliers: the pivot value is broadcast, 1/pivot formed once (or the
//      entries divided when |pivot| < DBL_MIN), and the kl multipliers reach
//      every lane by readlane (H <= 6) or by an LDS broadcast (H > 6);
//   4. lanes whose column is in j+1..ju apply one fma per window row;
//   5. every lane stores row j of the column that owns that register element
//      and refills the element with row j+H of its next column from a
//      prefetch ring PF steps deep.
// All memory traffic uses range-checked buffer operations and lane predicates
// are selects, so each unrolled step is straight-line code and the prefetch
// ring stays in flight.  The result is bitwise that of the unblocked
// algorithm: every entry sees the same fused multiply-adds in the same order.
#pragma once

#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"
#include "getrf_win2.hpp"
#include "getrf_lean64.hpp"

namespace bandlu {

// DPP lane permutation of a double (both halves moved with the same control)
#define BANDLU_DPP_D(v, ctrl)                                                                  \
    __longlong_as_double(                                                                      \
        ((long long)__builtin_amdgcn_mov_dpp((int)(__double_as_longlong(v) >> 32), ctrl, 0xf,  \
                                             0xf, false)                                       \
         << 32) |                                                                              \
        (unsigned)__builtin_amdgcn_mov_dpp((int)(__double_as_longlong(v) & 0xffffffffll), ctrl, \
                                           0xf, 0xf, false))

constexpr int pow2ceil(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// max over each row of 16 lanes (only the first H lanes of a row matter)
template <int H>
__device__ __forceinline__ double row_max16(double k) {
    k = fmax(k, BANDLU_DPP_D(k, 0xB1));   // quad_perm [1,0,3,2]
    if constexpr (H > 2) k = fmax(k, BANDLU_DPP_D(k, 0x4E));   // quad_perm [2,3,0,1]
    if constexpr (H > 4) k = fmax(k, BANDLU_DPP_D(k, 0x141));  // row_half_mirror
    if constexpr (H > 8) k = fmax(k, BANDLU_DPP_D(k, 0x140));  // row_mirror
    return k;
}

// The H window rows of one column as register vectors of at most 16 doubles:
// a wave-uniform dynamic index into such a vector becomes indexed register
// moves; longer vectors would be lowered through scratch memory.
template <int H>
struct WinCol {
    static constexpr int NV = H > 16 ? 2 : 1;
    static constexpr int VL = H > 16 ? 16 : pow2ceil(H);
    typedef double vec __attribute__((ext_vector_type(VL)));
    vec v[NV];
    // k is a compile-time constant after inlining
    __device__ __forceinline__ double get(int k) const {
        if (NV == 1 || k < 16) return v[0][k];
        return v[1][k - 16];
    }
    __device__ __forceinline__ void set(int k, double x) {
        if (NV == 1 || k < 16) v[0][k] = x;
        else v[1][k - 16] = x;
    }
    // k is wave-uniform
    __device__ __forceinline__ double dget(int k) const {
        if constexpr (NV == 1) return v[0][k];
        double r;
        if (k < 16) r = v[0][k];
        else r = v[1][k - 16];
        return r;
    }
    __device__ __forceinline__ void dset(int k, double x) {
        if constexpr (NV == 1) {
            v[0][k] = x;
        } else {
            if (k < 16) v[0][k] = x;
            else v[1][k - 16] = x;
        }
    }
};

template <int H, int CPL, int PF>
__global__ __launch_bounds__(64) void getrf_win64_kernel(WinParams P) {
    static_assert(PF % H == 0, "prefetch depth must be a multiple of H");
    static_assert(H <= 32, "window taller than 32 rows");
    constexpr int M = 64 * CPL;
    constexpr int kl = H - 1;
    constexpr bool TR = H > 6;
    const int L = threadIdx.x;
    const int64_t b = blockIdx.x;  // one matrix per workgroup (= wavefront)
    const int n = P.n, ku = P.ku, kv = kl + P.ku, ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + b * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    const Buf pb = make_buf(P.ipiv + b * P.strideP, uint32_t(int64_t(n) * 4));
    __shared__ double s_col[TR ? 32 : 1];
    __shared__ double s_l[TR ? 32 : 1];

    auto colof = [&](int s, int x) -> int { return x + (((L + 64 * s) - x) & (M - 1)); };
    auto foff = [&](int r, int c) -> uint32_t {  // original band entry (r, c), else outside
        const bool ok = c >= 0 && c < n && r >= 0 && r < n && unsigned(r - c + ku) <= unsigned(kl + ku);
        return ok ? uint32_t(c * ldab + kv + r - c) * 8u : kOutside;
    };

    WinCol<H> a[CPL];
    double pf[CPL][PF];
#pragma unroll
    for (int s = 0; s < CPL; ++s) {
#pragma unroll
        for (int r = 0; r < H; ++r) a[s].set(r, buf_ld(ab, foff(r, colof(s, r - H + 1))));
#pragma unroll
        for (int k = 0; k < PF; ++k) pf[s][k] = buf_ld(ab, foff(k + H, colof(s, k + 1)));
    }
    int ju = 0, info = 0;

    auto step = [&]<int U>(int j) __attribute__((always_inline)) {
        constexpr int S0 = U % H;
        const bool live = j < n;
        const int km = min(kl, n - 1 - j);
        const int src = j & 63;
        const int sj = (j >> 6) & (CPL - 1);
        int c[CPL];
#pragma unroll
        for (int s = 0; s < CPL; ++s) c[s] = colof(s, j);
        // ---- 1. pivot search
        int p = 0;
        double piv0 = 0.0;  // entry (j+p, j) before the interchange
        double x = 0.0;     // TR: row j+L of column j
        if constexpr (H > 1) {
            if constexpr (TR) {
                // the pivot lane writes its register elements in element order
                // (consecutive registers, wide LDS stores); lane t reads the
                // element of row j+t, i.e. element (S0 + t) mod H
                if (L == src) {
#pragma unroll
                    for (int k = 0; k < H; ++k) {
                        double v = a[0].get(k);
#pragma unroll
                        for (int s = 1; s < CPL; ++s) v = sj == s ? a[s].get(k) : v;
                        s_col[k] = v;
                    }
                }
                __builtin_amdgcn_wave_barrier();
                {
                    const int t = L & 31;
                    const int k = S0 + t < H ? S0 + t : S0 + t - H;
                    x = s_col[k < H ? k : 0];
                }
                double key = __builtin_isnan(x) ? (L == 0 ? __builtin_inf() : -1.0) : fabs(x);
                key = L <= km ? key : -2.0;
                double kmax = row_max16<H>(key);
                if constexpr (H > 16) {
                    const double k0 = readlane_d(kmax, 0), k1 = readlane_d(kmax, 16);
                    kmax = fmax(k0, k1);
                }
                const unsigned long long hit = __ballot(key == kmax);
                p = __builtin_amdgcn_readfirstlane(__builtin_ctzll(hit));
                piv0 = readlane_d(x, p);
            } else {
                double best = 0.0, bv = 0.0;
                int pl = 0;
#pragma unroll
                for (int s = 0; s < CPL; ++s) {
                    double b = fabs(a[s].get(S0));
                    double v0 = a[s].get(S0);
                    int ps = 0;
#pragma unroll
                    for (int t = 1; t < H; ++t) {
                        const double v = a[s].get((S0 + t) % H);
                        const bool gt = t <= km && fabs(v) > b;
                        b = gt ? fabs(v) : b;
                        v0 = gt ? v : v0;
                        ps = gt ? t : ps;
                    }
                    if (s == 0 || sj == s) { best = b; bv = v0; pl = ps; }
                }
                (void)best;
                p = __builtin_amdgcn_readlane(pl, src);
                piv0 = readlane_d(bv, src);
            }
        } else {
            double v = a[0].get(S0);
#pragma unroll
            for (int s = 1; s < CPL; ++s) v = sj == s ? a[s].get(S0) : v;
            piv0 = readlane_d(v, src);
        }
        const bool nz = live && piv0 != 0.0;
        buf_st_i32(pb, (L == 0 && live) ? uint32_t(j) * 4u : kOutside, j + p + 1);
        double lt = x;  // TR: this lane's multiplier (unscaled when the pivot is zero)
        if (nz) {
            ju = max(ju, min(j + ku + p, n - 1));
            // ---- 2. interchange rows j and j+p in columns j..ju
            if constexpr (H > 1) {
                if (p != 0) {
                    const int sp = S0 + p >= H ? S0 + p - H : S0 + p;
#pragma unroll
                    for (int s = 0; s < CPL; ++s) {
                        const bool m = c[s] <= ju;
                        const double x0 = a[s].get(S0);
                        const double xp = a[s].dget(sp);
                        a[s].set(S0, m ? xp : x0);
                        a[s].dset(sp, m ? x0 : xp);
                    }
                }
            }
            if constexpr (H > 1) {
                // ---- 3. multipliers
                const double piv = piv0;
                const bool big = fabs(piv) >= DBL_MIN;
                const double rcp = 1.0 / piv;
                double Lm[H];
                if constexpr (TR) {
                    const double x0 = readlane_d(x, 0);
                    const double xs = L == p ? x0 : (L == 0 ? piv : x);
                    lt = big ? xs * rcp : xs / piv;
                    lt = L == 0 ? piv : lt;
                    if (L < 32) s_l[L] = lt;  // lanes 32..63 mirror 0..31: one writer per slot
                    __builtin_amdgcn_wave_barrier();
#pragma unroll
                    for (int t = 1; t < H; ++t) Lm[t] = s_l[t];
                } else {
#pragma unroll
                    for (int t = 1; t < H; ++t) {
                        double v = a[0].get((S0 + t) % H);
#pragma unroll
                        for (int s = 1; s < CPL; ++s) v = sj == s ? a[s].get((S0 + t) % H) : v;
                        const double l = big ? v * rcp : v / piv;
                        Lm[t] = readlane_d(l, src);
                    }
#pragma unroll
                    for (int s = 0; s < CPL; ++s)
                        if (c[s] == j) {
#pragma unroll
                            for (int t = 1; t < H; ++t) a[s].set((S0 + t) % H, Lm[t]);
                        }
                }
                // ---- 4. rank-1 update of columns j+1..ju
#pragma unroll
                for (int s = 0; s < CPL; ++s) {
                    const bool m = c[s] > j && c[s] <= ju;
                    const double u = a[s].get(S0);
#pragma unroll
                    for (int t = 1; t < H; ++t) {
                        const double v = a[s].get((S0 + t) % H);
                        const double nv = __builtin_fma(-Lm[t], u, v);
                        a[s].set((S0 + t) % H, m ? nv : v);
                    }
                }
            }
        } else if (live && info == 0) {
            info = j + 1;
        }
        // ---- 5. stores and refill (straight-line, range-checked)
        if constexpr (TR) {  // multipliers of column j straight from the transposed lanes
            const bool ok = live && L >= 1 && L <= km;
            buf_st(ab, ok ? uint32_t(j * ldab + kv + L) * 8u : kOutside, lt);
        }
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
            const int co = colof(s, j - H + 1);
            const bool ok = live && co >= 0 && co < n && j >= co - kv && (!TR || co >= j);
            buf_st(ab, ok ? uint32_t(co * ldab + kv + j - co) * 8u : kOutside, a[s].get(S0));
            a[s].set(S0, pf[s][U]);
            pf[s][U] = buf_ld(ab, foff(j + PF + H, colof(s, j + PF + 1)));
        }
    };

    for (int j0 = 0; j0 < n; j0 += PF) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) {
            (step.template operator()<Us>(j0 + Us), ...);
        }(std::make_integer_sequence<int, PF>{});
    }
    if (L == 0) P.info[b] = info;
}

// kl <= 7: the wave-uniform pivot kernel (getrf_lean64.hpp); beyond, one
// column per lane with a transposed pivot column (getrf_win2.hpp), and the
// in-lane pivot scan for two columns per lane.
template <int H, int CPL>
constexpr WinKernel win64_pick() {
    if constexpr (H <= 8) return &getrf_lean64_kernel<H, CPL>;
    else if constexpr (CPL == 1) return &getrf_win2_kernel<H, win_pf(H)>;
    else return &getrf_win64_kernel<H, CPL, win_pf(H)>;
}

template <int CPL, int LO, int HI>
struct Win64Range {
    template <int... Is>
    static constexpr auto make(std::integer_sequence<int, Is...>) {
        return std::array<WinKernel, HI - LO + 1>{{win64_pick<LO + Is, CPL>()...}};
    }
};

}  // namespace bandlu
