// Banded LU with partial pivoting (xGBTRF semantics) for narrow bands
// (1 <= kl <= 31, 2kl+ku+1 <= 64 CPL), one matrix per workgroup of two
// wavefronts: the single-matrix kernel of Sec. III-A's specialised algorithm
// f(N).
//
// The column steps form one chain of dependent pivot decisions.  A single
// wavefront that also carries the rank-1 updates, the row stores and the
// refills issues a few hundred instructions per step, and one wavefront issues
// at most one instruction every four cycles.  Here the work of a step is split
// between two wavefronts that run on different SIMDs:
//   wave P (pivots) holds the pivot column transposed, one row per lane.  At
//     step j it takes column j (rows j-1..j-1+kl, up to date through step j-2)
//     from wave U, applies step j-1 to it (interchange, one fused multiply-add
//     per row) and adds the row that enters, finds the pivot (first largest
//     |a|; a NaN counts only in first position), forms the multipliers in the
//     lanes of their rows, stores ipiv[j], and hands the pivot offset and the
//     multipliers to wave U;
//   wave U (updates) runs one step behind with the band window in registers:
//     column c in lane (c mod M) mod 64, register sub-slot (c mod M) / 64
//     (M = 64 CPL), row r in slot r mod H (H = kl + 1).  At its step j it
//     applies the interchange and the rank-1 update of step j-1 to the window
//     columns, stores row j-1 of U and the multipliers of column j-1, refills
//     the freed slot with the row that enters, and hands column j+1 (rows
//     j..j+kl, up to date through step j-1) to wave P.  Wave U is the only
//     wave that writes the band array: wave P reads original entries only, and
//     each of them before wave U reaches the column that holds it.
// The two hand-overs are double buffered in LDS and one workgroup barrier per
// step separates them.  Every entry sees the same operations in the same order
// as in the unblocked algorithm, so the factors are bitwise those of the
// reference loops.
#pragma once

#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"
#include "wave.hpp"

namespace bandlu {

// 64-bit lane masks on the scalar unit: `len` lanes from lane `start` on,
// wrapping around (0 <= len <= 63)
__device__ __forceinline__ unsigned long long split_lanes(int start, int len) {
    const unsigned long long ones = (1ull << len) - 1;
    const int s = start & 63;
    return (ones << s) | ((ones >> 1) >> (63 - s));
}

// rotate right by r (0 <= r <= 63)
__device__ __forceinline__ unsigned long long split_rotr(unsigned long long m, int r) {
    return (m >> r) | ((m << 1) << (63 - r));
}

__device__ __forceinline__ unsigned split_wave_max(unsigned v) {
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xf, 0xf, false));
    v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xf, 0xf, false));
    const unsigned a = max((unsigned)__builtin_amdgcn_readlane((int)v, 0), (unsigned)__builtin_amdgcn_readlane((int)v, 16));
    const unsigned b = max((unsigned)__builtin_amdgcn_readlane((int)v, 32), (unsigned)__builtin_amdgcn_readlane((int)v, 48));
    return max(a, b);
}

// prefetch depth of wave U: an even multiple of H (so that the LDS buffer
// parity and every register slot index are compile-time constants), at least 16
constexpr int split_pf(int H) {
    int m = (16 + H - 1) / H;
    if ((m * H) & 1) ++m;
    return m * H;
}

template <int H, int CPL>
__global__ __launch_bounds__(128) void getrf_split_kernel(WinParams P) {
    constexpr int PF = split_pf(H);
    static_assert(H >= 2 && H <= 32, "window of 2..32 rows");
    static_assert(PF % H == 0 && PF % 2 == 0, "prefetch depth must be an even multiple of H");
    constexpr int M = 64 * CPL;
    constexpr int kl = H - 1;
    const int tid = threadIdx.x;
    const int L = tid & 63;
    const int64_t b = blockIdx.x;  // one matrix per workgroup
    const int ku = P.ku, kv = kl + P.ku, ldab = int(P.ldab);
    int n = P.n;
    double *ABb = P.AB + b * P.strideAB;
    int32_t *ipb = P.ipiv + b * P.strideP;
    int j0 = 0;
    if (P.resume) {
        // after the diagonal-pivot kernel (getrf_diag.hpp): ipiv[n-1] > 0 says
        // it factored the whole band, -(j0+1) that column j0 failed its check.
        // Steps 0..j0-1 interchanged nothing, so the trailing band from column
        // j0 on is a band problem of its own with the same kl and ku.
        const int m = ipb[n - 1];
        if (m > 0) return;
        j0 = -m - 1;
        n -= j0;
        ABb += int64_t(j0) * ldab;
        ipb += j0;
    }
    const Buf ab = make_buf(ABb, uint32_t(int64_t(ldab) * n * 8));
    __shared__ double s_l[2][32];    // multipliers of a step by row offset 1..kl
    __shared__ int s_pv[2][2];       // pivot offset and nonzero-pivot flag of a step
    __shared__ double s_col[2][64];  // a column for wave P, rows by offset from its first

    // original band entry (r, c), else an offset outside the buffer (reads 0)
    auto foff = [&](int r, int c) -> uint32_t {
        const bool ok = c >= 0 && c < n && r >= 0 && r < n && unsigned(r - c + ku) <= unsigned(kl + ku);
        return ok ? uint32_t(c * ldab + kv + r - c) * 8u : kOutside;
    };

    if (tid >= 64) {
        // ------------------------------------------------------------ wave U --
        auto colof = [&](int s, int x) -> int { return x + (((L + 64 * s) - x) & (M - 1)); };
        double a[CPL][H];
        double pf[CPL][PF];
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
#pragma unroll
            for (int r = 0; r < H; ++r) a[s][r] = buf_ld(ab, foff(r, colof(s, r - H + 1)));
#pragma unroll
            for (int k = 0; k < PF; ++k) pf[s][k] = buf_ld(ab, foff(k + H, colof(s, k + 1)));
        }
        int ju = 0;
        // column 1, rows 0..kl (no step applied yet) for wave P's step 1: it
        // sits in lane 1, slots 0..kl
        if (L == 1) {
#pragma unroll
            for (int t = 0; t < H; ++t) s_col[0][t] = a[0][t];
        }
        lds_barrier();
        bool live = true;
        auto ustep = [&]<int U>(int jj) __attribute__((always_inline)) {
            constexpr int S0 = U % H;
            constexpr int par = U & 1;  // jj & 1 (PF is even)
            if (!live) return;
            if (jj >= n) {
                live = false;
                return;
            }
            // ---- step jj as decided by wave P
            const int pv = s_pv[par][0];
            const int nz = s_pv[par][1];
            int c[CPL];
#pragma unroll
            for (int s = 0; s < CPL; ++s) c[s] = colof(s, jj);
            if (nz) {
                ju = max(ju, min(jj + ku + pv, n - 1));
                if (pv != 0) {
                    // interchange rows jj and jj+pv in columns jj..ju
#pragma unroll
                    for (int s = 0; s < CPL; ++s)
                        if (c[s] <= ju) win_swap<H, S0>(a[s], pv);
                }
                double lm[H];
#pragma unroll
                for (int t = 1; t < H; ++t) lm[t] = s_l[par][t];
                // rank-1 update of columns jj+1..ju, under an exec mask (the empty
                // volatile asm keeps the block a branch: as selects it would cost
                // two more instructions per entry)
#pragma unroll
                for (int s = 0; s < CPL; ++s) {
                    if (c[s] > jj && c[s] <= ju) {
                        const double uu = a[s][S0];
#pragma unroll
                        for (int t = 1; t < H; ++t)
                            a[s][(S0 + t) % H] = __builtin_fma(-lm[t], uu, a[s][(S0 + t) % H]);
                        asm volatile("" ::: "memory");
                    }
                }
            }
            // ---- multipliers of column jj (as wave P formed them; for a zero pivot
            // the column as it is) into the band: wave U is the only wave that
            // writes the band, so no store can overtake one of its loads of an
            // original entry
            {
                const int kmj = min(kl, n - 1 - jj);
                const double lv = s_l[par][L & 31];
                buf_st(ab, (L >= 1 && L <= kmj) ? uint32_t(jj * ldab + kv + L) * 8u : kOutside, lv);
            }
            // ---- row jj of U leaves the window (columns jj..jj+kv), row jj+H enters
#pragma unroll
            for (int s = 0; s < CPL; ++s) {
                const int co = colof(s, jj - H + 1);  // column owning slot S0 (retired ones are skipped)
                const bool ok = co >= jj && co < n && co <= jj + kv;
                buf_st(ab, ok ? uint32_t(co * ldab + kv + jj - co) * 8u : kOutside, a[s][S0]);
                a[s][S0] = pf[s][U];
                pf[s][U] = buf_ld(ab, foff(jj + PF + H, colof(s, jj + PF + 1)));
            }
            // ---- column jj+2, rows jj+1..jj+1+kl (through step jj), for wave P
            if (jj + 2 < n) {
                const int wc = (jj + 2) & (M - 1);
                if (L == (wc & 63)) {
                    if (CPL == 1 || wc < 64) {
#pragma unroll
                        for (int t = 0; t < H; ++t) s_col[par ^ 1][t] = a[0][(S0 + 1 + t) % H];
                    } else {
#pragma unroll
                        for (int t = 0; t < H; ++t) s_col[par ^ 1][t] = a[CPL - 1][(S0 + 1 + t) % H];
                    }
                }
            }
            if (jj + 1 < n) lds_barrier();
        };
        for (int jj0 = 0; live; jj0 += PF) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (ustep.template operator()<Us>(jj0 + Us), ...);
            }(std::make_integer_sequence<int, PF>{});
        }
        return;
    }

    // -------------------------------------------------------------- wave P --
    const Buf pb = make_buf(ipb, uint32_t(int64_t(n) * 4));
    // entering entries a(c+kl, c) of the 64 columns of this and the next block
    double E = buf_ld(ab, foff(L + kl, L));
    double En = buf_ld(ab, foff(64 + L + kl, 64 + L));
    // column 0, rows 0..kl
    double y = buf_ld(ab, L <= kl ? foff(L, 0) : kOutside);
    double lprev = 0.0;
    int pprev = 0, nzprev = 0, juprev = 0;
    int ju = 0, info = 0;
    for (int j = 0; j < n; ++j) {
        const int u = j & 63;
        if (j > 0) {
            // column j, rows j-1..j-1+kl through step j-2, from wave U
            const int q = (j - 1) & 63;  // lane of row j-1
            double v = s_col[(j - 1) & 1][(L - q) & 63];
            if (nzprev && j <= juprev) {
                // step j-1 on column j: interchange, then one fma per row below
                if (pprev != 0) {
                    const int qp = (q + pprev) & 63;
                    const double vq = readlane_d(v, q), vp = readlane_d(v, qp);
                    v = L == q ? vp : (L == qp ? vq : v);
                }
                const double u0 = readlane_d(v, q);
                const int kmp = min(kl, n - j);
                if (__builtin_amdgcn_inverse_ballot_w64(split_lanes(q + 1, kmp)))
                    v = __builtin_fma(-lprev, u0, v);
            }
            // row j+kl enters the window (no step has touched it yet)
            const double e = readlane_d(E, u);
            y = L == ((j + kl) & 63) ? e : v;
        }
        // ---- pivot: first largest |y| over rows j..j+km.  The maximum is taken
        // over the high 32 bits of |y|; a NaN on the diagonal ranks above
        // everything and one below it with the zeros, so an earlier row wins
        // against it; only rows that tie on the high word compare low words.
        const int km = min(kl, n - 1 - j);
        const unsigned long long cand = split_lanes(u, km + 1);
        const double rall = 1.0 / y;
        const bool nan = __builtin_isnan(y);
        const bool inc = __builtin_amdgcn_inverse_ballot_w64(cand);
        const int toff = (L - u) & 63;
        const unsigned yhi = unsigned(__double_as_longlong(y) >> 32) & 0x7fffffffu;
        const unsigned khi = !inc ? 0u : (nan ? (toff == 0 ? 0x7ff00001u : 0u) : yhi);
        unsigned long long hit = __ballot(khi == split_wave_max(khi)) & cand;
        if (__popcll(hit) > 1) {
            const bool tied = (hit >> L) & 1;
            const unsigned klo = (tied && !nan) ? unsigned(__double_as_longlong(y)) : 0u;
            hit &= __ballot(klo == split_wave_max(klo));
        }
        const int p = __builtin_ctzll(split_rotr(hit, u));
        const int lp = (u + p) & 63;
        const double piv = readlane_d(y, lp);
        const double rcp = readlane_d(rall, lp);  // 1/piv, formed beside the reduction
        buf_st_i32(pb, L == 0 ? uint32_t(j) * 4u : kOutside, j0 + j + p + 1);
        const bool nzj = piv != 0.0;
        // the interchange (none for a zero pivot: then every candidate is zero
        // and p = 0)
        const double y0 = readlane_d(y, u);
        y = L == u ? piv : (L == lp ? y0 : y);
        // multipliers; a zero pivot eliminates nothing and the column below the
        // diagonal stays as it is
        double l = nzj ? y * rcp : y;
        if (nzj && !(fabs(piv) >= DBL_MIN)) l = y / piv;
        if (nzj) ju = max(ju, min(j + ku + p, n - 1));
        if (!nzj && info == 0) info = j + 1;
        // ---- hand-over to wave U (which also stores the multipliers)
        const bool mrow = __builtin_amdgcn_inverse_ballot_w64(split_lanes(u + 1, km));
        if (mrow) s_l[j & 1][toff] = l;
        if (L == 0) {
            s_pv[j & 1][0] = p;
            s_pv[j & 1][1] = nzj ? 1 : 0;
        }
        lprev = l;
        pprev = p;
        nzprev = nzj ? 1 : 0;
        juprev = ju;
        lds_barrier();
        if (u == 63) {
            E = En;
            En = buf_ld(ab, foff(j + 65 + L + kl, j + 65 + L));
        }
    }
    if (L == 0) {
        if (!P.resume) P.info[b] = info;
        else if (info != 0 && P.info[b] == 0) P.info[b] = j0 + info;
    }
}

// kernels of one CPL for H = LO..HI
template <int CPL, int LO, int HI>
struct SplitRange {
    template <int... Is>
    static constexpr auto make(std::integer_sequence<int, Is...>) {
        return std::array<WinKernel, HI - LO + 1>{{&getrf_split_kernel<LO + Is, CPL>...}};
    }
};

WinKernel split_kernel_c1_h2_16(int H);
WinKernel split_kernel_c1_h17_32(int H);
WinKernel split_kernel_c2_h2_16(int H);

}  // namespace bandlu
