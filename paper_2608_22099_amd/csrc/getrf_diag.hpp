// Banded LU for narrow bands that first assumes every pivot is the diagonal
// entry: the common case of Sec. III-A's specialised algorithm f(N), with
// xGBTRF semantics kept exactly.
//
// Partial pivoting keeps the diagonal entry of column j whenever no entry
// below it has a larger pivot key (ties go to the diagonal).  While that
// holds, the factorisation has no row interchanges, no fill-in beyond the
// ku superdiagonals and no cross-lane argmax; each column step is
//   piv = u(j,j);  l(i) = a(i,j) * (1/piv);  a(i,c) -= l(i) * u(j,c),
// for i = j+1..j+kl and c = j+1..j+ku, with the operations (reciprocal,
// product, fused multiply-add) and their order exactly those of the
// unblocked pivoting algorithm, so the factors are bitwise its factors.
// Every step checks that no candidate row outranks the diagonal before it
// changes anything.  The first column j0 that fails ends the kernel: it writes
// the band as it stands before step j0 and marks ipiv[n-1] = -(j0+1).  The
// two-wavefront pivoting kernel then factors the trailing band from column j0
// on as a problem of its own (getrf_split.hpp): steps 0..j0-1 interchanged
// nothing, and the product-form L of xGBTRF never moves earlier multipliers.
//
// One wavefront per matrix.  Row r lives in lane r mod 64 from the step at
// which its first entry enters the window until the step that stores its last
// one; its entries sit in register slots by column, column c in slot
// c mod (ku+2).  The original band reaches the wavefront in chunks of C
// consecutive columns: one batch of 16-byte loads per chunk, issued a chunk
// ahead into staging registers and copied into an LDS buffer (double
// buffered) when the chunk begins, so no step waits on global memory.  A
// step j
//   - takes u(j,j) and 1/u(j,j) from the lane of row j with lane reads into
//     scalar registers, and checks the kl candidates, exiting on the first
//     failure;
//   - takes the rest of row j, u(j,j+1..j+ku), as vector registers: every
//     lane writes its row to LDS at the end of a step and the next pivot row
//     is read back at once as a broadcast, so the read is in flight during
//     the step boundary (two lane reads per entry cost more);
//   - reads column j+ku+1 from the chunk buffer into the slot column j-1 has
//     left, each lane its own row;
//   - forms the multipliers and the rank-1 update in the lanes of rows
//     j+1..j+kl, ku fused multiply-adds per lane, column j+1 first: row
//     j+1 is then final and its lane forms 1/u(j+1,j+1), one stage of the
//     division between every one or two of the other updates;
//   - stores column j of the factors (U entries kept in their rows' lanes
//     since those rows were pivot rows, the multipliers, and zeros in the
//     fill slots): one coalesced store.
// The lane masks of a step live in scalar registers, so its control never
// waits for a vector result, except for the one test of the candidates.
// One chunk of steps is unrolled, so that every register index is a
// compile-time constant; chunks away from both ends of the matrix run a copy
// without the bounds tests.
#pragma once

#include <array>
#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"

namespace bandlu {

// steps per chunk for upper bandwidth KU: a multiple of the slot period, at
// least 16 and no longer than that needs (every step of a chunk is unrolled,
// and longer chunks no longer fit the instruction cache)
constexpr int diag_chunk(int KU) { return (KU + 2) * ((16 + KU + 1) / (KU + 2)); }
// Largest kl for KU: the live rows (from j-KU, whose U entries are still to
// be stored, to j+KU+1+kl, the last row column j+KU+1 reaches) need a lane
// each, and the 2kl+KU+1 rows a column store covers must fall in distinct
// lanes.
constexpr int diag_max_kl(int KU) {
    const int a = 62 - 2 * KU, b = (63 - KU) / 2;
    return a < b ? a : b;
}
constexpr int kDiagMaxKu = 24;

typedef unsigned diag_v4u __attribute__((ext_vector_type(4)));

// 1/v by the hardware's correctly rounded division sequence (scale, reciprocal
// estimate, two Newton refinements, quotient correction, fix-up of special
// operands), one instruction per stage, so that a caller can place other work
// between the dependent stages; bitwise the quotient 1.0 / v.
struct DiagRecip {
    double den, d, nn, r, e, q;
    bool flag;
    template <int G>
    __device__ __forceinline__ void stage() {
        if constexpr (G == 0) {
            bool f0;
            d = __builtin_amdgcn_div_scale(1.0, den, false, &f0);
            nn = __builtin_amdgcn_div_scale(1.0, den, true, &flag);
        } else if constexpr (G == 1) {
            r = __builtin_amdgcn_rcp(d);
        } else if constexpr (G == 2) {
            e = __builtin_fma(-d, r, 1.0);
        } else if constexpr (G == 3) {
            r = __builtin_fma(r, e, r);
        } else if constexpr (G == 4) {
            e = __builtin_fma(-d, r, 1.0);
        } else if constexpr (G == 5) {
            r = __builtin_fma(r, e, r);
        } else if constexpr (G == 6) {
            q = nn * r;
        } else if constexpr (G == 7) {
            e = __builtin_fma(-d, q, nn);
        } else if constexpr (G == 8) {
            q = __builtin_amdgcn_div_fmas(e, r, q, flag);
        } else {
            q = __builtin_amdgcn_div_fixup(q, den, 1.0);
        }
    }
    static constexpr int kStages = 10;
};

template <int KU>
__global__ __launch_bounds__(64) void getrf_diag_kernel(WinParams P) {
    constexpr int S = KU + 2;               // window slots: columns j-1..j+KU
    constexpr int C = diag_chunk(KU);       // steps (and band columns) per chunk
    constexpr int NST = (C * 64) / 128 + 1;  // 16-byte loads per lane for a chunk (ldab <= 64)
    constexpr int G = 64;                   // guard doubles on both sides of a chunk buffer
    const int L = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int n = P.n, kl = P.kl, kv = kl + KU, ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + b * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    int32_t *const ipiv = P.ipiv + b * P.strideP;
    // original band columns of a chunk, laid out as in memory (ldab apart),
    // with guard zones: every lane reads its slot without a bounds test
    __shared__ double s_col[2][G + C * 64 + G];
    // every lane's row after a step (entry k of the row at [k][lane]), read
    // back whole by the next step for its pivot row
    __shared__ double s_u[KU + 1][64];

    for (int j = L; j < n - 1; j += 64) ipiv[j] = j + 1;

    // chunk k holds band columns k*C+KU+1 .. k*C+KU+C, which enter the window
    // at steps k*C .. k*C+C-1
    const int cbytes = C * ldab * 8;
    diag_v4u stg[NST];
    auto stage = [&](int k) __attribute__((always_inline)) {
        const uint32_t base = uint32_t(k * C + KU + 1) * uint32_t(ldab) * 8u;
#pragma unroll
        for (int i = 0; i < NST; ++i) {
            const int o = (i * 64 + L) * 16;
            stg[i] = __builtin_amdgcn_raw_buffer_load_b128(ab.r, o < cbytes ? base + uint32_t(o) : kOutside,
                                                           0, 0);
        }
    };
    auto commit = [&](int k) __attribute__((always_inline)) {
        char *dst = reinterpret_cast<char *>(s_col[k & 1] + G);
#pragma unroll
        for (int i = 0; i < NST; ++i) {
            const int o = (i * 64 + L) * 16;
            if (o < cbytes) *reinterpret_cast<diag_v4u *>(dst + o) = stg[i];
        }
    };

    // at step s lane L holds row s + eof(s), eof(s) in [-KU, 63-KU]
    auto eof = [&](int s) { return ((L - s + KU) & 63) - KU; };
    double x[S];
    double un[KU + 1];  // the next step's pivot row, u(j+1, j+1..j+1+KU)
    {
        const int r = eof(0);
#pragma unroll
        for (int c = 0; c <= KU; ++c) {
            const int d = r - c;
            const bool ok = c < n && r >= 0 && r < n && d >= -KU && d <= kl;
            x[c] = buf_ld(ab, ok ? uint32_t(c * ldab + kv + d) * 8u : kOutside);
        }
        x[S - 1] = 0.0;
#pragma unroll
        for (int k = 1; k <= KU; ++k) s_u[k][L] = x[k];
#pragma unroll
        for (int k = 1; k <= KU; ++k) un[k] = s_u[k][0];
        stage(0);
        commit(0);
        stage(1);
    }
    // lane masks of step s, relative to the lane of row s and rotated by one
    // lane per step
    auto low = [](int k) -> unsigned long long { return k >= 64 ? ~0ull : (1ull << k) - 1; };
    auto rotr = [](unsigned long long m, int k) -> unsigned long long {
        return k == 0 ? m : (m >> k) | (m << (64 - k));
    };
    unsigned long long m_act = low(kl) << 1;               // rows s+1..s+kl
    unsigned long long m_up = rotr(low(KU + kl + 1), KU);  // rows s-KU..s+kl
    unsigned long long m_st = rotr(low(kv + kl + 1), kv);  // rows s-kv..s+kl (column s store)
    double rn = 1.0 / x[0];  // lane of row s: 1/u(s,s) once step s-1 has run
    int info = 0;
    int stop = -1;  // the first column whose diagonal entry would not be the pivot
    const double *cur = s_col[0] + G;
    // step s; false once the factorisation stops (a failed check, or s = n)
    auto step = [&]<bool EDGE, int Q>(int s) __attribute__((always_inline)) -> bool {
        constexpr int X = Q % S;  // slot of column s
        if (EDGE && s >= n) return false;
        const int e = eof(s);
        const int ls = s & 63;
        unsigned long long act = m_act, st = m_st;
        if (EDGE) {
            // near either end of the matrix: rows outside it take no part
            const int rs = e <= kl ? s + e : s + e - 64;
            act &= __builtin_amdgcn_ballot_w64(s + e < n);
            st &= __builtin_amdgcn_ballot_w64(rs >= 0 && rs < n);
        }
        const double piv = readlane_d(x[X], ls);
        // a candidate with a larger key than the diagonal's: an ordered
        // comparison of magnitudes is that test, NaNs included (a NaN
        // candidate ranks last, a NaN diagonal first)
        if (__builtin_amdgcn_ballot_w64(fabs(x[X]) > fabs(piv)) & act) {
            stop = s;
            return false;
        }
        double u[KU + 1];
#pragma unroll
        for (int k = 1; k <= KU; ++k) u[k] = un[k];
        // column s+KU+1 enters the window, in the slot column s-1 has left
        // (lanes of other rows read a harmless entry: no row uses its slot
        // for that column)
        x[(X + S - 1) % S] = cur[Q * ldab + kv + e - (KU + 1)];
        const double rcp = readlane_d(rn, ls);
        double l = x[X] * rcp;
        const unsigned hi = unsigned(__double_as_longlong(piv) >> 32);
        if (__builtin_expect(((hi >> 20) & 0x7ffu) - 1u >= 0x7feu, 0)) {
            // zero, below DBL_MIN, infinite or NaN: the pivoting loop's choices
            if (piv == 0.0) {
                act = 0;  // nothing to eliminate
                if (info == 0) info = s + 1;
            } else if (!(fabs(piv) >= DBL_MIN)) {
                l = x[X] / piv;
            }
        }
        // Row s+1 is final once column s+1 is updated: its lane forms the
        // next reciprocal at once, each stage of the division followed by a
        // share of the other columns' updates, which do not depend on it.
        // With nothing to eliminate (a zero pivot) it is formed on its own.
        if (__builtin_amdgcn_inverse_ballot_w64(act)) {
            x[X] = l;
            x[(X + 1) % S] = __builtin_fma(-l, u[1], x[(X + 1) % S]);
            DiagRecip dv;
            dv.den = x[(X + 1) % S];
            [&]<int... Gs>(std::integer_sequence<int, Gs...>) __attribute__((always_inline)) {
                (
                    [&] {
                        dv.template stage<Gs>();
                        constexpr int NF = KU - 1, NG = DiagRecip::kStages;
#pragma unroll
                        for (int f = Gs * NF / NG; f < (Gs + 1) * NF / NG; ++f)
                            x[(X + 2 + f) % S] = __builtin_fma(-l, u[2 + f], x[(X + 2 + f) % S]);
                        __builtin_amdgcn_sched_barrier(0);
                    }(),
                    ...);
            }(std::make_integer_sequence<int, DiagRecip::kStages>{});
            rn = dv.q;
            asm volatile("" ::: "memory");  // keep the block a branch under an exec mask
        }
        if (__builtin_expect(act == 0, 0)) rn = 1.0 / x[(X + 1) % S];
        // this lane's row as it now stands; the lane of row s+1 holds the
        // next pivot row, read back at once (a broadcast) for the next step
#pragma unroll
        for (int k = 1; k <= KU; ++k) s_u[k][L] = x[(X + 1 + k) % S];
#pragma unroll
        for (int k = 1; k <= KU; ++k) un[k] = s_u[k][(s + 1) & 63];
        // column s of the factors: U rows s-KU..s, multipliers s+1..s+kl, and
        // zeros in the fill slots of rows s-kv..s-KU-1 (those lanes belong to
        // rows 64 further on, which column s does not reach)
        {
            const bool up = __builtin_amdgcn_inverse_ballot_w64(m_up);
            const int rel = up ? e : e - 64;  // row minus s
            const uint32_t voff = __builtin_amdgcn_inverse_ballot_w64(st) ? uint32_t(kv + rel) * 8u : kOutside;
            buf_st_so(ab, voff, uint32_t(s * ldab) * 8u, up ? x[X] : 0.0);
        }
        m_act = rotr(m_act, 63);
        m_up = rotr(m_up, 63);
        m_st = rotr(m_st, 63);
        if constexpr (Q == C - 1) {
            // the next chunk into LDS (its loads were issued a chunk ago),
            // and the loads of the one after it. Here, not after the chunk:
            // only a chunk that ran all its steps gets here, so the wait for
            // the loads counts this chunk's column stores as issued after
            // them (where the early exits join, it waits for those too).
            const int k = (s - (C - 1)) / C;
            commit(k + 1);
            stage(k + 2);
        }
        return true;
    };
    auto chunk = [&]<bool EDGE>(int s0) __attribute__((always_inline)) -> bool {
        return [&]<int... Qs>(std::integer_sequence<int, Qs...>) __attribute__((always_inline)) {
            return (step.template operator()<EDGE, Qs>(s0 + Qs) && ...);
        }(std::make_integer_sequence<int, C>{});
    };
    for (int s0 = 0;; s0 += C) {
        const int k = s0 / C;
        cur = s_col[k & 1] + G;
        const bool interior = s0 >= kv && s0 + C + KU + kl + 1 <= n;
        const bool go = interior ? chunk.template operator()<false>(s0) : chunk.template operator()<true>(s0);
        if (!go || s0 + C >= n) break;
    }
    if (stop >= 0) {
        // the band as it stands before step `stop`: entries that earlier steps
        // changed and no column store has written (rows up to stop+kl-1 in
        // columns stop..stop+KU-1, U rows above included) ...
        const int s = stop;
        const int r = s + eof(s);
#pragma unroll
        for (int q = 0; q < S; ++q) {
            const int c = s + ((q - s) % S + S) % S;  // the column in slot q (s-1 counts as s+KU+1)
            const bool ok = c <= s + KU - 1 && c < n && r >= 0 && r >= c - KU && r <= s + kl - 1;
            buf_st(ab, ok ? uint32_t(c * ldab + kv + r - c) * 8u : kOutside, x[q]);
        }
        // ... and zeros in the fill slots of rows above `stop` in the columns
        // they reach
        for (int c = s; c < n && c < s + kv; ++c) {
            const int rf = c - kv + L;
            const bool ok = L < kl && rf >= 0 && rf < s && rf < c - KU;
            buf_st(ab, ok ? uint32_t(c * ldab + L) * 8u : kOutside, 0.0);
        }
        if (L == 0) ipiv[n - 1] = -(s + 1);
    } else if (L == 0) {
        ipiv[n - 1] = n;
    }
    if (L == 0) P.info[b] = info;
}


template <int LO, int HI>
struct DiagRange {
    template <int... Is>
    static constexpr auto make(std::integer_sequence<int, Is...>) {
        return std::array<WinKernel, HI - LO + 1>{{&getrf_diag_kernel<LO + Is>...}};
    }
};

WinKernel diag_kernel_ku1_8(int KU);
WinKernel diag_kernel_ku9_16(int KU);
WinKernel diag_kernel_ku17_24(int KU);

}  // namespace bandlu
