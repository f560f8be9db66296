// Banded LU with partial pivoting (xGBTRF semantics) for one matrix per
// wavefront and kl <= 7: the register-window form of Sec. III-A's specialised
// algorithm f(N) with the pivot decided as a wave-uniform value.
//
// Layout.  Column c lives in lane ((c mod M) / CPL), sub-slot c mod CPL,
// M = 64 * CPL >= 2kl+ku+1; row r of a column lives in register slot r mod 16.
// The step loop is unrolled by 16, so every slot index, and the sub-slot of
// the pivot column, is a compile-time constant.
//
// Step j:
//   1. the kl+1 window rows of column j reach every lane by lane reads into
//      scalar registers; the pivot (first largest |a|, a NaN counts only in
//      first position: every comparison with it is false) and its offset p
//      are then decided on scalars, so p is wave-uniform;
//   2. the interchange of rows j and j+p is one uniform branch on p, a select
//      per lane whose column is in j..ju;
//   3. every lane forms the same reciprocal and multipliers from the scalars
//      (a division per entry when |pivot| < DBL_MIN), and the lane of column j
//      keeps them in its slots;
//   4. lanes whose column is in j+1..ju apply one fma per window row;
//   5. every lane stores row j of the column that owns that slot (U row j for
//      active columns, a multiplier for retired ones) and refills the slot of
//      row j+kl+1 from a prefetch ring 16 steps deep.
// The operations and their order are those of the unblocked algorithm, so
// the factors are bitwise equal to it.
//
// FWD: the forward half of the solve (xGBTRS's L y = P b, one right-hand side)
// runs in the same steps: rows j..j+kl of b are wave-uniform values in a
// 16-slot ring; step j interchanges rows j and j+p, keeps y(j), and step j+1
// applies step j's
//   b(j+t) = fma(-l(j+t,j), y(j), b(j+t)),  t = 1..kl,
// with the multipliers as stored (the raw column for a zero pivot), as the
// plain forward loop does.  Rows enter from two registers that hold a block
// of 16 rows each in lanes 0..15; y leaves one block at a time.  Blocks of 16 steps away from both
// ends (every index in range, kl candidates at every step) address memory
// with a per-lane offset plus one scalar offset and test no ranges; the
// blocks at the ends check every index.
#pragma once

#include <cfloat>
#include <utility>

#include "bufio.hpp"
#include "common.hpp"
#include "getrf_window.hpp"

namespace bandlu {

template <int H, int CPL, bool FWD = false>
__global__ __launch_bounds__(64) void getrf_lean64_kernel(WinParams P) {
    static_assert(H >= 1 && H <= 8, "kl <= 7");
    static_assert(CPL == 1 || CPL == 2, "one or two columns per lane");
    constexpr int kl = H - 1;
    constexpr int PF = 16;
    constexpr int M = 64 * CPL;
    const int L = threadIdx.x;
    const int64_t b = blockIdx.x;  // one matrix per workgroup (= wavefront)
    const int ku = P.ku, kv = kl + P.ku, ldab = int(P.ldab);
    int n = P.n;
    double *ABb = P.AB + b * P.strideAB;
    int32_t *ipb = P.ipiv + b * P.strideP;
    int jr = 0;  // first column of this launch (resume mode)
    if (P.resume) {
        // after the diagonal-pivot kernel (getrf_diag.hpp): ipiv[n-1] > 0 says
        // it factored the whole band, -(j0+1) that column j0 failed its check.
        // Steps 0..j0-1 interchanged nothing, so the trailing band from column
        // j0 on is a band problem of its own with the same kl and ku.
        const int m = ipb[n - 1];
        if (m > 0) return;
        jr = -m - 1;
        n -= jr;
        ABb += int64_t(jr) * ldab;
        ipb += jr;
    }
    const Buf ab = make_buf(ABb, uint32_t(int64_t(ldab) * n * 8));
    const Buf pb = make_buf(ipb, uint32_t(int64_t(n) * 4));

    // the column in [x, x + M) held by sub-slot s of this lane
    auto colof = [&](int s, int x) -> int { return x + ((CPL * L + s - x) & (M - 1)); };
    // original band entry (r, c), else outside
    auto foff = [&](int r, int c) -> uint32_t {
        const bool ok = c >= 0 && c < n && r >= 0 && r < n && unsigned(r - c + ku) <= unsigned(kv);
        return ok ? uint32_t(c * ldab + kv + r - c) * 8u : kOutside;
    };
    // Lean blocks: at step j sub-slot s stores row j of column j + e and loads
    // row j + 16 + H of column j + 17 + f, where
    //   e + H - 1 = (CPL*L + s + H - 1 - j) mod M   (stored while e <= kv),
    //   f         = (CPL*L + s - 17 - j) mod M      (in the band while f <= ku + H - 1).
    // Both offsets are a per-lane part plus the scalar (j - 16) * ldab * 8; lean
    // blocks start at j >= 16, which keeps every per-lane part positive.
    const uint32_t stride8 = uint32_t(ldab - 1) * 8u;
    const uint32_t st_base = uint32_t(16 * ldab + kv - (H - 1) * (ldab - 1)) * 8u;
    const uint32_t ld_base = uint32_t(33 * ldab + kv + H - 1) * 8u;

    double a[CPL][16];
    double pf[CPL][PF];
#pragma unroll
    for (int s = 0; s < CPL; ++s) {
#pragma unroll
        for (int r = 0; r < 16; ++r) a[s][r] = r < H ? buf_ld(ab, foff(r, colof(s, r - H + 1))) : 0.0;
#pragma unroll
        for (int k = 0; k < PF; ++k) pf[s][k] = buf_ld(ab, foff(k + H, colof(s, k + 1)));
    }
    int ju = 0, info = 0;
    int pv = 0;  // lane U < 16: the 1-based pivot row of this block's step U

    // forward solve: rows of b by slot r mod 16, the block's rows and the
    // next block's in lanes 0..15, y(j) of step U in lane U
    const Buf bb = make_buf(FWD ? P.B + b * P.strideB : P.AB, FWD ? uint32_t(n) * 8u : 0u);
    double bw[16], bcur = 0.0, bnext = 0.0, yv = 0.0;
    double lp[H], yp = 0.0;  // the last step's multipliers (as stored) and y
#pragma unroll
    for (int t = 0; t < H; ++t) lp[t] = 0.0;
    if constexpr (FWD) {
        bcur = buf_ld(bb, L < PF ? uint32_t(L) * 8u : kOutside);
        bnext = buf_ld(bb, L < PF ? uint32_t(PF + L) * 8u : kOutside);
#pragma unroll
        for (int r = 0; r < H; ++r) bw[r] = own_copy(readlane_d(bcur, r));
    }

    auto step = [&]<int U, bool LEAN>(int j) __attribute__((always_inline)) {
        constexpr int S0 = U;              // slot of row j
        constexpr int SJ = U & (CPL - 1);  // sub-slot of column j (blocks start at multiples of 16)
        const int km = LEAN ? kl : min(kl, n - 1 - j);
        const int lo = (j / CPL) & 63;     // the lane of column j
        // ---- 1. pivot: every lane scans its sub-slot SJ column the same way
        // and the lane of column j gives the offset and the value
        double bl = a[SJ][S0];
        int pl = 0;
#pragma unroll
        for (int t = 1; t < H; ++t) {
            const double v = a[SJ][(S0 + t) & 15];
            const bool gt = (LEAN || t <= km) && fabs(v) > fabs(bl);  // false for a NaN
            bl = gt ? v : bl;
            pl = gt ? t : pl;
        }
        // column j's window rows before the interchange, as scalars
        double cv[H];
#pragma unroll
        for (int t = 0; t < H; ++t) cv[t] = readlane_d(a[SJ][(S0 + t) & 15], lo);
        const int p = __builtin_amdgcn_readlane(pl, lo);
        const double best = readlane_d(bl, lo);
        pv = L == U ? jr + j + p + 1 : pv;
        // A zero pivot (every candidate zero) leaves the step without an
        // interchange (p = 0), a multiplier or an update: the masks below
        // carry nz instead of a branch.
        const bool nz = best != 0.0;
        info = (!nz && info == 0) ? j + 1 : info;
        ju = nz ? max(ju, LEAN ? j + ku + p : min(j + ku + p, n - 1)) : ju;
        const int span = ju - j;
        // relative column c - j of each sub-slot, in [0, M)
        int d[CPL];
#pragma unroll
        for (int s = 0; s < CPL; ++s) d[s] = (CPL * L + s - j) & (M - 1);
        double cs[H], lm[H], old[CPL][H];
        bool upd[CPL], own = false;
        if constexpr (H > 1) {
            // ---- 2. interchange rows j and j+p in columns j..ju (selects)
#pragma unroll
            for (int s = 0; s < CPL; ++s) {
                const bool m = d[s] <= span;
                const double x0 = a[s][S0];
                double xp = a[s][(S0 + 1) & 15];
#pragma unroll
                for (int k = 2; k < H; ++k) xp = p == k ? a[s][(S0 + k) & 15] : xp;
                a[s][S0] = (m && p != 0) ? xp : x0;
#pragma unroll
                for (int k = 1; k < H; ++k)
                    a[s][(S0 + k) & 15] = (m && p == k) ? x0 : a[s][(S0 + k) & 15];
            }
            // ---- 3. multipliers, the same in every lane
#pragma unroll
            for (int t = 1; t < H; ++t) cs[t] = p == t ? cv[0] : cv[t];
            const double rcp = 1.0 / best;
#pragma unroll
            for (int t = 1; t < H; ++t) lm[t] = cs[t] * rcp;
            own = nz && L == lo;
#pragma unroll
            for (int t = 1; t < H; ++t) a[SJ][(S0 + t) & 15] = own ? lm[t] : a[SJ][(S0 + t) & 15];
            // ---- 4. rank-1 update of columns j+1..ju (the entries before it
            // are kept for the rare pivot below DBL_MIN)
#pragma unroll
            for (int s = 0; s < CPL; ++s) {
                upd[s] = nz && unsigned(d[s] - 1) < unsigned(span);
                const double u = a[s][S0];
#pragma unroll
                for (int t = 1; t < H; ++t) {
                    old[s][t] = a[s][(S0 + t) & 15];
                    const double nv = __builtin_fma(-lm[t], u, old[s][t]);
                    a[s][(S0 + t) & 15] = upd[s] ? nv : old[s][t];
                }
            }
        }
        // ---- 5. row j leaves; row j+H enters its slot from the prefetch ring
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
            if constexpr (LEAN) {
                const uint32_t soff = uint32_t(j - 16) * uint32_t(ldab) * 8u;
                const uint32_t es = uint32_t(CPL * L + s + H - 1 - j) & uint32_t(M - 1);
                const uint32_t fs = uint32_t(CPL * L + s + M - 17 - j) & uint32_t(M - 1);
                const uint32_t sto = es <= uint32_t(kv + H - 1) ? __umul24(es, stride8) + st_base : kOutside;
                const uint32_t ldo = fs <= uint32_t(ku + H - 1) ? __umul24(fs, stride8) + ld_base : kOutside;
                buf_st_so(ab, sto, soff, a[s][S0]);
                a[s][(S0 + H) & 15] = own_copy(pf[s][U]);
                pf[s][U] = buf_ld_so(ab, ldo, soff);
            } else {
                const int co = colof(s, j - H + 1);
                const bool ok = co >= 0 && co < n && j >= co - kv;
                buf_st(ab, ok ? uint32_t(co * ldab + kv + j - co) * 8u : kOutside, a[s][S0]);
                a[s][(S0 + H) & 15] = own_copy(pf[s][U]);
                pf[s][U] = buf_ld(ab, foff(j + PF + H, colof(s, j + PF + 1)));
            }
        }
        if constexpr (H > 1) {
            // A pivot below DBL_MIN (a NaN or zero one too; the masks ignore
            // the multipliers of a zero pivot) divides instead: the update is
            // redone from the kept entries.  Placed last, this one rare branch
            // leaves the rest of the step in one scheduling region.
            if (__builtin_expect(!(fabs(best) >= DBL_MIN), 0)) {
                // (a zero pivot leaves its column as it is: the forward solve
                // then reads the multipliers as stored, the raw column)
#pragma unroll
                for (int t = 1; t < H; ++t) lm[t] = nz ? cs[t] / best : cv[t];
#pragma unroll
                for (int t = 1; t < H; ++t) a[SJ][(S0 + t) & 15] = own ? lm[t] : a[SJ][(S0 + t) & 15];
#pragma unroll
                for (int s = 0; s < CPL; ++s) {
                    const double u = a[s][S0];
#pragma unroll
                    for (int t = 1; t < H; ++t)
                        a[s][(S0 + t) & 15] =
                            upd[s] ? __builtin_fma(-lm[t], u, old[s][t]) : a[s][(S0 + t) & 15];
                }
            }
        }
        if constexpr (FWD) {
            // ---- forward solve, one step behind: the update of step j-1
            // (its multipliers and y(j-1) are at hand, so these instructions
            // wait for nothing on this step's chain), then the interchange of
            // step j and y(j); step j's update waits for step j+1
            if constexpr (H > 1) {
#pragma unroll
                for (int t = 1; t < H; ++t)
                    bw[(S0 + t - 1) & 15] = __builtin_fma(-lp[t], yp, bw[(S0 + t - 1) & 15]);
            }
            const double b0 = bw[S0];
            double bj = b0;
            if constexpr (H > 1) {
                double bp = bw[(S0 + 1) & 15];
#pragma unroll
                for (int k = 2; k < H; ++k) bp = p == k ? bw[(S0 + k) & 15] : bp;
                bj = p != 0 ? bp : b0;
#pragma unroll
                for (int k = 1; k < H; ++k) bw[(S0 + k) & 15] = p == k ? b0 : bw[(S0 + k) & 15];
#pragma unroll
                for (int t = 1; t < H; ++t) lp[t] = own_copy(lm[t]);  // the column as stored
            }
            yp = own_copy(bj);
            yv = L == U ? bj : yv;
            // row j+H enters (step j's update, applied at step j+1, reaches
            // rows j+1..j+kl only).  The b window, the last multipliers and y
            // sit in vector registers (own_copy): as scalars they crowd out
            // the step's scalar registers, which then spill to vector lanes.
            bw[(S0 + H) & 15] =
                own_copy(U + H < PF ? readlane_d(bcur, (U + H) & 15) : readlane_d(bnext, (U + H) & 15));
        }
    };

    auto block = [&]<bool LEAN>(int j0) __attribute__((always_inline)) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) __attribute__((always_inline)) {
            if constexpr (LEAN) {
                (step.template operator()<Us, true>(j0 + Us), ...);
            } else {
                ((j0 + Us < n ? step.template operator()<Us, false>(j0 + Us) : (void)0), ...);
            }
        }(std::make_integer_sequence<int, PF>{});
        buf_st_i32(pb, (L < PF && j0 + L < n) ? uint32_t(j0 + L) * 4u : kOutside, pv);
        if constexpr (FWD) {
            buf_st(bb, (L < PF && j0 + L < n) ? uint32_t(j0 + L) * 8u : kOutside, yv);
            bcur = own_copy(bnext);
            bnext = buf_ld(bb, (L < PF && j0 + 2 * PF + L < n) ? uint32_t(j0 + 2 * PF + L) * 8u : kOutside);
        }
    };

    // lean block: stores of columns >= 0 (j0 >= 16 > H - 1), loads of rows and
    // columns < n, and kl candidates at every step.  The lean blocks run in a
    // loop of their own, so the prefetch ring's loads carry their true age
    // across the loop's back edge and each step waits only for its own row.
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
    if (L == 0) {
        if (!P.resume) P.info[b] = info;
        else if (info != 0 && P.info[b] == 0) P.info[b] = jr + info;
    }
}

}  // namespace bandlu
