// Banded LU with partial pivoting (xGBTRF semantics) with the active window
// held in registers: Sec. III-A's specialised algorithm f(N), for narrow bands.
//
// A group of G lanes (G = 64: one matrix per wavefront; G = 16: four matrices
// per wavefront, all at the same step) factors one matrix.  At step j the
// active window is rows j..j+kl by columns j..j+kl+ku.  Column c lives in
// lane (c mod M) mod G, register sub-slot (c mod M) / G, where M = G * CPL;
// row r of a column lives in register slot r mod H (H = kl + 1).  Because the
// step loop is unrolled by a multiple of H, every register index is a
// compile-time constant.  Each step:
//   1. the lane holding column j finds the pivot (first largest |a|, a NaN
//      is taken only in first position) and broadcasts p;
//   2. lanes whose column is in j..ju swap register slots j and j+p;
//   3. the pivot lane scales its column by 1/pivot (or divides when
//      |pivot| < DBL_MIN) and broadcasts the kl multipliers;
//   4. lanes whose column is in j+1..ju apply one fma per window row;
//   5. every lane stores row j of the column that owns that register slot
//      (U row j for active columns, a multiplier for retired ones), then
//      refills the slot with row j+H of its next column from a prefetch ring
//      that runs PF steps ahead.
// So each lane issues exactly one load and one store per step, and every
// in-matrix slot of the band array is written exactly once, at the step of its
// row.  M >= 2kl+ku+1 guarantees that a lane's slots are refilled with zeros
// (fill rows) before it takes a new column.
#pragma once

#include <array>
#include <cfloat>
#include <utility>

#include "common.hpp"

namespace bandlu {

struct WinParams {
    double *AB;
    int32_t *ipiv;
    int32_t *info;
    int64_t ldab, strideAB, strideP;
    int n, ku, batch;
    int kl;      // read by the kernels that take kl at run time
    int resume;  // two-wavefront and lean window kernels: continue where the diagonal-pivot kernel stopped
    // lean window kernel with the forward solve: one right-hand side per
    // matrix, B + b * strideB (set only for that kernel)
    double *B = nullptr;
    int64_t strideB = 0;
};

template <int G>
__device__ __forceinline__ int win_bcast_i(int v, int src) {
    if constexpr (G == 64) return __builtin_amdgcn_readlane(v, src);
    else return __shfl(v, src, G);
}

template <int G>
__device__ __forceinline__ double win_bcast_d(double v, int src) {
    if constexpr (G == 64) {
        long long x = __double_as_longlong(v);
        int lo = __builtin_amdgcn_readlane((int)(x & 0xffffffffll), src);
        int hi = __builtin_amdgcn_readlane((int)(x >> 32), src);
        return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
    } else {
        return __shfl(v, src, G);
    }
}

// swap slots S0 and (S0 + p) % H for a runtime p in [1, H): a chain of
// selects, so the register array is never indexed dynamically (a dynamic index
// would push the whole window out to scratch memory)
template <int H, int S0>
__device__ __forceinline__ void win_swap(double (&a)[H], int p) {
    double a0 = a[S0];
#pragma unroll
    for (int k = 1; k < H; ++k) {
        const bool hit = p == k;
        const double ak = a[(S0 + k) % H];
        a0 = hit ? ak : a0;
        a[(S0 + k) % H] = hit ? a[S0] : ak;
    }
    a[S0] = a0;
}

template <int H, int G, int CPL, int PF>
__global__ __launch_bounds__(64) void getrf_window_kernel(WinParams P) {
    static_assert(PF % H == 0, "prefetch depth must be a multiple of H");
    constexpr int M = G * CPL;
    constexpr int kl = H - 1;
    const int lane = threadIdx.x;
    const int gl = lane & (G - 1);
    const int b = blockIdx.x * (64 / G) + lane / G;
    const bool live = b < P.batch;
    double *__restrict__ AB = P.AB + (live ? int64_t(b) * P.strideAB : 0);
    int32_t *__restrict__ ipiv = P.ipiv + (live ? int64_t(b) * P.strideP : 0);
    const int n = P.n, ku = P.ku, kv = kl + P.ku;
    const int64_t ldab = P.ldab;

    // column held by sub-slot s at step x: smallest c >= x with c == slot (mod M)
    auto colof = [&](int s, int x) -> int { return x + (((gl + s * G) - x) & (M - 1)); };
    // original band entry (row r, column c), +0.0 for fill rows and outside
    auto fetch = [&](int r, int c) -> double {
        const bool ok = live && c >= 0 && c < n && r >= 0 && r < n && r >= c - ku && r <= c + kl;
        return ok ? AB[int64_t(c) * ldab + (kv + r - c)] : 0.0;
    };

    double a[CPL][H];
    double pf[CPL][PF];
#pragma unroll
    for (int s = 0; s < CPL; ++s) {
#pragma unroll
        for (int r = 0; r < H; ++r) a[s][r] = fetch(r, colof(s, r - H + 1));
#pragma unroll
        for (int k = 0; k < PF; ++k) pf[s][k] = fetch(k + H, colof(s, k + 1));
    }
    int ju = 0, info = 0;

    auto step = [&]<int U>(int j) {
        constexpr int S0 = U % H;
        const int km = min(kl, n - 1 - j);
        const int src = j & (G - 1);
        int c[CPL];
#pragma unroll
        for (int s = 0; s < CPL; ++s) c[s] = colof(s, j);
        // 1. pivot search on each sub-slot; the pivot lane's sub-slot is used
        int pinfo = 0;
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
            double best = fabs(a[s][S0]);
            int p = 0;
#pragma unroll
            for (int t = 1; t < H; ++t) {
                const double v = fabs(a[s][(S0 + t) % H]);
                if (t <= km && v > best) { best = v; p = t; }
            }
            const int pi = p | (best != 0.0 ? 0 : 256);
            if (s == 0 || c[s] == j) pinfo = pi;
        }
        pinfo = win_bcast_i<G>(pinfo, src);
        const int p = pinfo & 255;
        const bool zero = (pinfo >> 8) != 0;
        if (live && gl == src) ipiv[j] = j + p + 1;
        if (!zero) {
            ju = max(ju, min(j + ku + p, n - 1));
            // 2. interchange rows j and j+p in columns j..ju
            if constexpr (H > 1) {
                if (p != 0) {
#pragma unroll
                    for (int s = 0; s < CPL; ++s)
                        if (c[s] <= ju) win_swap<H, S0>(a[s], p);
                }
            }
            double pv = a[0][S0];
#pragma unroll
            for (int s = 1; s < CPL; ++s) if (c[s] == j) pv = a[s][S0];
            const double piv = win_bcast_d<G>(pv, src);
            if constexpr (H > 1) {
                // 3. multipliers, formed in the pivot lane
                if (fabs(piv) >= DBL_MIN) {
                    const double rcp = 1.0 / piv;
#pragma unroll
                    for (int s = 0; s < CPL; ++s)
                        if (c[s] == j) {
#pragma unroll
                            for (int t = 1; t < H; ++t) a[s][(S0 + t) % H] = a[s][(S0 + t) % H] * rcp;
                        }
                } else {
#pragma unroll
                    for (int s = 0; s < CPL; ++s)
                        if (c[s] == j) {
#pragma unroll
                            for (int t = 1; t < H; ++t) a[s][(S0 + t) % H] = a[s][(S0 + t) % H] / piv;
                        }
                }
                double L[H];
#pragma unroll
                for (int t = 1; t < H; ++t) {
                    double lv = a[0][(S0 + t) % H];
#pragma unroll
                    for (int s = 1; s < CPL; ++s) if (c[s] == j) lv = a[s][(S0 + t) % H];
                    L[t] = win_bcast_d<G>(lv, src);
                }
                // 4. rank-1 update of columns j+1..ju
#pragma unroll
                for (int s = 0; s < CPL; ++s) {
                    if (c[s] > j && c[s] <= ju) {
                        const double u = a[s][S0];
#pragma unroll
                        for (int t = 1; t < H; ++t)
                            a[s][(S0 + t) % H] = __builtin_fma(-L[t], u, a[s][(S0 + t) % H]);
                    }
                }
            }
        } else if (info == 0) {
            info = j + 1;
        }
        // 5. store row j of the column owning slot S0, refill the slot
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
            const int co = colof(s, j - H + 1);
            if (live && co >= 0 && co < n && j >= co - kv)
                AB[int64_t(co) * ldab + (kv + j - co)] = a[s][S0];
            a[s][S0] = pf[s][U];
            pf[s][U] = fetch(j + PF + H, colof(s, j + PF + 1));
        }
    };

    for (int j0 = 0; j0 < n; j0 += PF) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) {
            ((j0 + Us < n ? step.template operator()<Us>(j0 + Us) : (void)0), ...);
        }(std::make_integer_sequence<int, PF>{});
    }
    if (live && gl == 0) P.info[b] = info;
}

// Prefetch depth: a multiple of H that reaches at least 16 steps ahead.
constexpr int win_pf(int H) { return H * ((16 + H - 1) / H); }

using WinKernel = void (*)(WinParams);

// Table of window kernels for H = LO..HI with fixed G and CPL.
template <int G, int CPL, int LO, int HI>
struct WinRange {
    template <int... Is>
    static constexpr auto make(std::integer_sequence<int, Is...>) {
        return std::array<WinKernel, HI - LO + 1>{
            {&getrf_window_kernel<LO + Is, G, CPL, win_pf(LO + Is)>...}};
    }
};

// Kernel for (G, CPL, H), or null if none is instantiated.
WinKernel win_kernel(int G, int CPL, int H);

}  // namespace bandlu
