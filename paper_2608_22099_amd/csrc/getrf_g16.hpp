// Batched banded LU with partial pivoting (xGBTRF semantics) for small
// bands: sixteen lanes per matrix, four matrices per wavefront, all four at
// the same column step (Sec. III-A's specialised algorithm f(N), the batched
// form).  kl <= 7 and 2kl+ku+1 <= 16.
//
// Lane i of a group holds column c == i (mod 16) of its matrix's band window;
// the window rows of that column live in sixteen register slots (row mod 16),
// of which kl+1 are active.  With the step loop unrolled by 16, the lane that
// holds column j and the slot of row j are compile-time constants, so the
// pivot, the pivot offset and the multipliers reach the other lanes of a
// group by one DPP row broadcast each (row_newbcast), with no LDS traffic.
// The four matrices pivot independently: the row interchange is a chain of
// selects on the group's pivot offset, and the update runs under a per-lane
// exec mask.  All loads and stores go through one range-checked buffer over
// the whole batch, so each step is branch-free and a 16-step prefetch ring
// stays in flight.  Every entry sees the same fused multiply-adds, in the same
// order, as in the unblocked algorithm.
//
// A single wavefront per SIMD runs the chain of steps, one instruction at a
// time, so the step's instruction count is its time.  Blocks of 16 steps away
// from both ends of the matrix (every index in range, kl candidates at every
// step) therefore take a lean step: no range tests, the load and store offsets
// of step U read from two per-lane tables (the part that grows with j is one
// scalar offset), and, when all four pivots are normal numbers, no zero-pivot
// or small-pivot handling.  The pivots of a block are kept in a register and
// stored once per block.
#pragma once

#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"

namespace bandlu {

// value of lane K of this lane's row of 16 (every lane is written, so the
// old value is the source itself: no separate zeroing of the destination)
template <int K>
__device__ __forceinline__ int row_bcast_i(int v) {
    return __builtin_amdgcn_update_dpp(v, v, 0x150 + K, 0xf, 0xf, false);
}

template <int K>
__device__ __forceinline__ double row_bcast_d(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = row_bcast_i<K>((int)(x & 0xffffffffll));
    const int hi = row_bcast_i<K>((int)(x >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

template <int H>
__global__ __launch_bounds__(64) void getrf_g16_kernel(WinParams P) {
    static_assert(H >= 1 && H <= 8, "kl <= 7");
    constexpr int kl = H - 1;
    constexpr int PF = 16;
    const int lane = threadIdx.x;
    const int gl = lane & 15;
    const int b = blockIdx.x * 4 + (lane >> 4);
    const bool live = b < P.batch;
    const unsigned long long livemask = __builtin_amdgcn_ballot_w64(live);
    const int n = P.n, ku = P.ku, kv = kl + P.ku, ldab = int(P.ldab);
    // one buffer over the whole batch (the host checks that it is < 2 GiB)
    const Buf ab = make_buf(P.AB, uint32_t(int64_t(P.batch) * P.strideAB * 8));
    const Buf pb = make_buf(P.ipiv, uint32_t(int64_t(P.batch) * P.strideP * 4));
    const uint32_t mbase = live ? uint32_t(int64_t(b) * P.strideAB * 8) : kOutside;
    const uint32_t pbase = live ? uint32_t(int64_t(b) * P.strideP * 4) : kOutside;

    // the column in [x, x+16) this lane holds
    auto colof = [&](int x) -> int { return x + ((gl - x) & 15); };
    // original band entry (r, c) of this lane's matrix, else outside
    auto foff = [&](int r, int c) -> uint32_t {
        const bool ok = c >= 0 && c < n && r >= 0 && r < n && unsigned(r - c + ku) <= unsigned(kv);
        return ok ? mbase + uint32_t(c * ldab + kv + r - c) * 8u : kOutside;
    };
    // The lean steps' offsets: at step j = 16m + U, row j leaves to column
    // co = j + d (d = ((gl + H - 1 - U) mod 16) - H + 1, stored while
    // d <= kv) and row j + 16 + H is loaded for column c = j + e
    // (e = 17 + ((gl - U - 1) mod 16), in the band while e <= ku + H + 16).
    // Both offsets are a per-lane part that depends on U only plus the scalar
    // (j - 16) * ldab * 8 (lean blocks have j >= 16, so that every per-lane
    // part, 16 * ldab + d * (ldab-1) + kv with d >= -7, is positive).
    uint32_t st_tab[16], ld_tab[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const int d = ((gl + H - 1 - u) & 15) - H + 1;
        st_tab[u] = d <= kv ? mbase + uint32_t(16 * ldab + d * (ldab - 1) + kv) * 8u : kOutside;
        const int e = 17 + ((gl - u - 1) & 15);
        ld_tab[u] = e <= ku + H + 16 ? mbase + uint32_t(16 * ldab + e * (ldab - 1) + kv + 16 + H) * 8u
                                     : kOutside;
    }

    double a[16];
    double pf[PF];
#pragma unroll
    for (int r = 0; r < 16; ++r) a[r] = r < H ? buf_ld(ab, foff(r, colof(r - H + 1))) : 0.0;
#pragma unroll
    for (int k = 0; k < PF; ++k) pf[k] = buf_ld(ab, foff(k + H, colof(k + 1)));
    int ju = 0, info = 0;
    int pv = 0;  // the 1-based pivot row of this block's step gl

    // steps 2..4 of the unblocked algorithm (interchange, multipliers,
    // update) for any pivot
    auto tail_any = [&]<int U>(int j, int p, double piv) __attribute__((always_inline)) {
        constexpr int S0 = U;
        const int c = colof(j);
        const bool elim = piv != 0.0;
        info = (!elim && info == 0) ? j + 1 : info;
        if (elim) {
            ju = max(ju, min(j + ku + p, n - 1));
            // ---- 2. interchange rows j and j+p in columns j..ju
            if constexpr (H > 1) {
                if (c <= ju) {
                    double a0 = a[S0];
#pragma unroll
                    for (int k = 1; k < H; ++k) {
                        const bool hit = p == k;
                        const double ak = a[(S0 + k) & 15];
                        a0 = hit ? ak : a0;
                        a[(S0 + k) & 15] = hit ? a[S0] : ak;
                    }
                    a[S0] = a0;
                }
                // ---- 3. multipliers, formed in the lane of column j
                if (gl == U) {
                    if (fabs(piv) >= DBL_MIN) {
                        const double rcp = 1.0 / piv;
#pragma unroll
                        for (int t = 1; t < H; ++t) a[(S0 + t) & 15] = a[(S0 + t) & 15] * rcp;
                    } else {
#pragma unroll
                        for (int t = 1; t < H; ++t) a[(S0 + t) & 15] = a[(S0 + t) & 15] / piv;
                    }
                }
                // ---- 4. rank-1 update of columns j+1..ju
                double lm[H];
#pragma unroll
                for (int t = 1; t < H; ++t) lm[t] = row_bcast_d<U>(a[(S0 + t) & 15]);
                if (c > j && c <= ju) {
                    const double uu = a[S0];
#pragma unroll
                    for (int t = 1; t < H; ++t) a[(S0 + t) & 15] = __builtin_fma(-lm[t], uu, a[(S0 + t) & 15]);
                }
            }
        }
    };

    auto step = [&]<int U, bool LEAN>(int j, uint32_t soff) __attribute__((always_inline)) {
        constexpr int S0 = U;  // slot of row j; lane U of each group holds column j
        const int km = LEAN ? kl : min(kl, n - 1 - j);
        // ---- 1. pivot: the lane of column j scans its kl+1 rows (first
        // largest |a|; a NaN counts only in first position: every comparison
        // with it is false), then its group takes the offset and the value
        double best = a[S0];
        int pl = 0;
#pragma unroll
        for (int t = 1; t < H; ++t) {
            const double v = a[(S0 + t) & 15];
            const bool gt = (LEAN || t <= km) && fabs(v) > fabs(best);  // false for a NaN
            best = gt ? v : best;
            pl = gt ? t : pl;
        }
        const int p = row_bcast_i<U>(pl);
        const double piv = row_bcast_d<U>(best);
        pv = gl == U ? j + p + 1 : pv;
        if constexpr (LEAN && H > 1) {
            // all four pivots normal numbers: no zero-pivot step, no division
            const bool normal = fabs(piv) >= DBL_MIN && fabs(piv) <= DBL_MAX;
            if ((__builtin_amdgcn_ballot_w64(!normal) & livemask) == 0ull) {
                const int c = j + ((gl - U) & 15);
                ju = max(ju, j + ku + p);
                const int pe = c <= ju ? p : 0;
                double a0 = a[S0];
#pragma unroll
                for (int k = 1; k < H; ++k) {
                    const bool hit = pe == k;
                    const double ak = a[(S0 + k) & 15];
                    a0 = hit ? ak : a0;
                    a[(S0 + k) & 15] = hit ? a[S0] : ak;
                }
                a[S0] = a0;
                if (gl == U) {
                    const double rcp = 1.0 / piv;
#pragma unroll
                    for (int t = 1; t < H; ++t) a[(S0 + t) & 15] = a[(S0 + t) & 15] * rcp;
                }
                double lm[H];
#pragma unroll
                for (int t = 1; t < H; ++t) lm[t] = row_bcast_d<U>(a[(S0 + t) & 15]);
                if (c > j && c <= ju) {
                    const double uu = a[S0];
#pragma unroll
                    for (int t = 1; t < H; ++t) a[(S0 + t) & 15] = __builtin_fma(-lm[t], uu, a[(S0 + t) & 15]);
                }
            } else {
                tail_any.template operator()<U>(j, p, piv);
            }
        } else {
            tail_any.template operator()<U>(j, p, piv);
        }
        // ---- 5. row j leaves (U row j for active columns, a multiplier for
        // retired ones); row j+H enters its slot from the prefetch ring
        if constexpr (LEAN) {
            buf_st_so(ab, st_tab[U], soff, a[S0]);
            a[(S0 + H) & 15] = own_copy(pf[U]);
            pf[U] = buf_ld_so(ab, ld_tab[U], soff);
        } else {
            const int co = colof(j - H + 1);
            const bool ok = co < n && j >= co - kv;
            buf_st(ab, ok ? mbase + uint32_t(co * ldab + kv + j - co) * 8u : kOutside, a[S0]);
            a[(S0 + H) & 15] = own_copy(pf[U]);
            pf[U] = buf_ld(ab, foff(j + PF + H, colof(j + PF + 1)));
        }
    };

    auto block = [&]<bool LEAN>(int j0) __attribute__((always_inline)) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) __attribute__((always_inline)) {
            if constexpr (LEAN) {
                (step.template operator()<Us, true>(j0 + Us, uint32_t(j0 + Us - PF) * uint32_t(ldab) * 8u), ...);
            } else {
                ((j0 + Us < n ? step.template operator()<Us, false>(j0 + Us, 0u) : (void)0), ...);
            }
        }(std::make_integer_sequence<int, PF>{});
        buf_st_i32(pb, j0 + gl < n ? pbase + uint32_t(j0 + gl) * 4u : kOutside, pv);
    };
    // lean block: stores of columns >= 0 (j0 >= 16 > H - 1), loads of rows
    // and columns < n, and kl candidates at every step.  The lean blocks run
    // in a loop of their own (no join with the other block's code at the
    // loop head, where every load in flight would be waited for).
    auto lean = [&](int j0) { return j0 >= PF && j0 + 2 * PF + kv + H < n; };
    for (int j0 = 0; j0 < n;) {
        if (lean(j0)) {
            do {
                block.template operator()<true>(j0);
                j0 += PF;
            } while (lean(j0));
        } else {
            block.template operator()<false>(j0);
            j0 += PF;
        }
    }
    if (live && gl == 0) P.info[b] = info;
}

}  // namespace bandlu
