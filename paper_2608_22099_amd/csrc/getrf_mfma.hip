// Blocked banded LU with partial pivoting whose trailing update runs on the
// fp64 matrix cores: the wide-band case of Sec. III-A's specialised algorithm
// f(N), with xGBTRF semantics for the factors, ipiv and info.
//
// Panels of NB = 32 columns, one launch per panel k.  Every workgroup of the
// launch takes a block of 32 band columns that panel k-1 reaches and applies
// that panel to it:
//   1. the panel's row interchanges, as one gather of the block's rows;
//   2. U12 = L11^-1 * (top 32 rows), one lane per column;
//   3. A22 += (-L21) * U12 with v_mfma_f64_16x16x4f64, four waves of 64 rows.
// Workgroup 0's block is panel k itself, which it then factors with partial
// pivoting: one thread per row, the row's 32 entries in registers, one LDS
// barrier per column step (every wave publishes its best candidate row and
// the diagonal row is published beside them, so the winner is known to all
// threads after the barrier without a second round trip).
//
// Multipliers are stored in xGBTRF's product form: the multipliers of column j
// stay in the rows they had when column j was eliminated, and later
// interchanges do not move them.  The blocked update needs L with the later
// interchanges of the panel applied; each workgroup rebuilds it from the
// stored multipliers and ipiv by tracing every row back through the panel's
// interchanges, so nothing but the band and ipiv passes between launches.
//
// Rounding differs from the unblocked order (the contraction sums in a
// different order), so the factors agree with the unblocked algorithm to
// rounding, not bitwise.
#include <algorithm>
#include <cfloat>
#include <climits>
#include <utility>

#include "common.hpp"
#include "wave.hpp"

namespace bandlu {

int launch_band_zero_fill(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int64_t strideAB, int32_t *d_info, int64_t batch, hipStream_t s);

int launch_getrf_mfma(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s);

namespace {

typedef double v4d __attribute__((ext_vector_type(4)));

constexpr int NB = 32;              // panel width = column block width
constexpr int kMaxKl = 256;
constexpr int kRows = NB + kMaxKl;  // rows a panel reaches
constexpr int kThreads = 320;       // five full waves; threads >= kRows only take part in barriers
constexpr int kWaves = kThreads / 64;
constexpr int LDX = NB + 1;         // row stride of the column block in LDS
constexpr int LDL = kRows + 8;      // column stride of the transposed panel L in LDS

struct MfmaParams {
    double *AB;
    int32_t *ipiv;
    int32_t *info;
    int64_t ldab, strideAB, strideP;
    int n, kl, ku;
    int j;           // first column of the panel applied (has_update)
    int jn;          // first column of workgroup 0's block: the panel factored
    int has_update;
};

__global__ __launch_bounds__(kThreads) void mfma_step_kernel(MfmaParams P) {
    const int bm = blockIdx.y;
    double *__restrict__ AB = P.AB + int64_t(bm) * P.strideAB;
    int32_t *__restrict__ ipiv = P.ipiv + int64_t(bm) * P.strideP;
    const int n = P.n, kl = P.kl, kv = P.kl + P.ku;
    const int64_t ldab = P.ldab;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const bool upd = P.has_update != 0;
    const bool fac = blockIdx.x == 0;
    const int jn = P.jn;
    const int cb = jn + int(blockIdx.x) * NB;  // first column of this block

    __shared__ double sX[kRows * LDX];   // block rows j .. j+R-1, after the interchanges
    __shared__ double sLT[NB * LDL];     // -L of the applied panel, transposed
    __shared__ int s_piv[NB];

    // ----------------------------------------------- apply panel k-1 --
    // (the panel applied always has NB columns: a narrower one is the last)
    const int j = P.j;
    const int R = upd ? min(NB + kl, n - j) : 0;
    const int W = upd ? min(NB, min(n, j + NB + kv) - cb) : 0;
    if (upd) {
        if (t < NB) s_piv[t] = ipiv[j + t] - 1 - (j + t);
        lds_barrier();
        if (t < kRows) {
            // trace band row j+t back through the panel's interchanges: src[s]
            // is where it was when column j+s was eliminated, pos where it was
            // before the panel
            int pos = j + t;
            int src[NB];
#pragma unroll
            for (int s = NB - 1; s >= 0; --s) {
                src[s] = pos;
                const int a = j + s, b = a + s_piv[s];
                pos = pos == a ? b : (pos == b ? a : pos);
            }
            // all loads first (conditions kept as bit fields), then the LDS writes
            double v[NB], u[NB];
            unsigned okv = 0, oku = 0;
#pragma unroll
            for (int s = 0; s < NB; ++s) {
                const int col = j + s;
                const int off = src[s] - col;
                const bool ok = (t < R) & (t > s) & (off >= 1) & (off <= min(kl, n - 1 - col));
                okv |= unsigned(ok) << s;
                v[s] = ld_clamped(AB, int64_t(col) * ldab + (kv + off), ok);
            }
#pragma unroll
            for (int c = 0; c < NB; ++c) {
                const int col = cb + c;
                const int d = pos - col;
                const bool ok = (t < R) & (c < W) & (d >= -kv) & (d <= kl);
                oku |= unsigned(ok) << c;
                u[c] = ld_clamped(AB, int64_t(col) * ldab + (kv + d), ok);
            }
#pragma unroll
            for (int s = 0; s < NB; ++s) sLT[s * LDL + t] = -keep_if(v[s], okv, s);
#pragma unroll
            for (int c = 0; c < NB; ++c) sX[t * LDX + c] = keep_if(u[c], oku, c);
        }
        lds_barrier();
        // U12 = L11^-1 * (rows 0..NB-1): wave 0, one lane per column
        if (wv == 0 && lane < NB) {
            double y[NB];
#pragma unroll
            for (int r = 0; r < NB; ++r) y[r] = sX[r * LDX + lane];
#pragma unroll
            for (int s = 0; s < NB - 1; ++s)
#pragma unroll
                for (int r = s + 1; r < NB; ++r) y[r] = __builtin_fma(sLT[s * LDL + r], y[s], y[r]);
#pragma unroll
            for (int r = 0; r < NB; ++r) sX[r * LDX + lane] = y[r];
        }
        lds_barrier();
        // rows NB..R-1 += (-L21) * U12 on the matrix cores.  Wave w < 4 owns
        // rows NB + 64w .. +63 as 4 x 2 tiles of 16 x 16.  Operand lanes of
        // v_mfma_f64_16x16x4f64: A[lane % 16][lane / 16], B[lane / 16][lane % 16];
        // accumulator element q of a lane is D[4q + lane / 16][lane % 16].
        if (wv < 4 && NB + 64 * wv < R) {
            const int r0 = NB + 64 * wv;
            const int ln = lane & 15, lk = lane >> 4;
            v4d acc[4][2];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        acc[rt][ct][q] = sX[(r0 + 16 * rt + 4 * q + lk) * LDX + 16 * ct + ln];
#pragma unroll
            for (int kb = 0; kb < NB / 4; ++kb) {
                const int k = 4 * kb + lk;
                const double b0 = sX[k * LDX + ln];
                const double b1 = sX[k * LDX + 16 + ln];
#pragma unroll
                for (int rt = 0; rt < 4; ++rt) {
                    const double a = sLT[k * LDL + r0 + 16 * rt + ln];
                    acc[rt][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b0, acc[rt][0], 0, 0, 0);
                    acc[rt][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b1, acc[rt][1], 0, 0, 0);
                }
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        sX[(r0 + 16 * rt + 4 * q + lk) * LDX + 16 * ct + ln] = acc[rt][ct][q];
        }
        lds_barrier();
        // write back: every row of a trailing block, only U12 for workgroup 0
        // (its other rows go on to the factorisation)
        const int rows = fac ? NB : R;
        if (t < rows) {
#pragma unroll
            for (int c = 0; c < NB; ++c) {
                const int col = cb + c;
                const int d = j + t - col;
                if (c < W && d >= -kv && d <= kl) AB[int64_t(col) * ldab + (kv + d)] = sX[t * LDX + c];
            }
        }
    }
    if (!fac) return;

    // ------------------------------------------------- factor panel k --
    // Each thread holds one band row of the panel: row jn + myrow, its 32
    // entries in registers.  An interchange does not move data: the thread
    // holding the pivot row takes the diagonal row's number and the diagonal
    // row's thread takes the pivot row's number.  The step loop runs in four
    // groups of eight columns; after each group the register row moves down by
    // eight (x[c] is column jn + 8g + c in group g), so every register index in
    // the loop body is a compile-time constant and the body is compiled once
    // per column of a group.
    __shared__ double sW[2][kWaves][NB];  // best candidate row of each wave
    __shared__ double sK[2][8];  // each wave's best key
    __shared__ double sR[2][8];  // and the reciprocal of its candidate pivot
    __shared__ int sI[2][8];     // and that candidate's row number
    const int nbn = min(NB, n - jn);
    const int Rn = min(nbn + kl, n - jn);
    const bool own = t < Rn;
    const int xr = NB + t;  // row of band row jn+t in the block above
    const bool from_lds = upd && xr < R;
    double x[NB];
    // band entry (row jn+t, column jn+c) is at diag0 + c * (ldab - 1); the
    // stride is hidden from the optimiser where it is used, so that the 32
    // column offsets are formed there and not kept live across the kernel
    const int64_t diag0 = int64_t(jn) * ldab + kv + t;
    auto colstep = [&]() __attribute__((always_inline)) {
        int64_t st = ldab - 1;
        asm volatile("" : "+s"(st));
        return st;
    };
    auto load_panel = [&]() __attribute__((always_inline)) {
        const int64_t st = colstep();
        unsigned okx = 0, okl = 0;
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            const int d = t - c;
            const bool inb = own & (c < nbn) & (d >= -kv) & (d <= kl);
            const bool lds = inb & from_lds & (c < W);
            okx |= unsigned(inb & !lds) << c;
            okl |= unsigned(lds) << c;
            x[c] = ld_clamped(AB, diag0 + c * st, inb & !lds);
        }
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            const double l = sX[min(xr, kRows - 1) * LDX + c];
            x[c] = (okl >> c & 1u) ? l : keep_if(x[c], okx, c);
        }
    };
    load_panel();

    // ---- first attempt: the panel with every pivot on the diagonal.  Partial
    // pivoting keeps the diagonal entry exactly when no candidate below it has
    // a larger pivot key (a tie goes to the first, the diagonal), so every
    // thread checks its row at every step instead of taking part in an argmax.
    // Without interchanges row s is final once steps 0..s-1 have reached it,
    // and the rows below need nothing but the pivot rows: wave 0 (rows 0..63)
    // runs the 32 steps, taking pivot row s from lane s with lane reads, and
    // publishes the pivot rows in groups of eight; the other waves apply each
    // group while wave 0 computes the next one.  Every entry gets its updates
    // in the order of the steps, with the operations of the pivoting loop
    // below, so the results are those of that loop whenever it would not
    // interchange.  Nothing is written before the whole panel has passed; if
    // any row outranks its diagonal, the panel is loaded again and factored by
    // the pivoting loop.
    constexpr int LDU = NB + 2;  // pivot row s: sU[s * LDU + c], c >= s; its reciprocal at c = NB
    double *const sU = sLT;      // (the applied panel's L is no longer needed)
    __shared__ int s_viol;
    bool viol = false;
    int finfo = 0;
    if (t == 0) s_viol = 0;
    const int ngrp = (nbn + 7) / 8;
    double r = 1.0 / x[0];  // wave 0: reciprocal of this row's entry in the next step's column
    double myrcp = 0.0;     // wave 0, lane s: the reciprocal of its pivot, once step s has run
    // step S in wave 0: pivot row S is lane S's row
    auto step_w0 = [&]<int S>() __attribute__((always_inline)) {
        if (S >= nbn) return;
        const double piv = readlane_d(x[S], S);
        const double rcp = readlane_d(r, S);
        myrcp = lane == S ? rcp : myrcp;
        const int km = min(kl, n - 1 - (jn + S));
        const int tt = t - S;
        const bool cand = own & (tt >= 1) & (tt <= km);
        viol |= cand && pivot_key(x[S], tt) > pivot_key(piv, 0);
        double u[NB];
#pragma unroll
        for (int c = S + 1; c < NB; ++c) u[c] = readlane_d(x[c], S);
        if (piv != 0.0) {
            double l;
            if (fabs(piv) >= DBL_MIN) {
                l = x[S] * rcp;
            } else {
                l = x[S] / piv;
            }
            if (cand) {
                x[S] = l;
#pragma unroll
                for (int c = S + 1; c < NB; ++c) x[c] = __builtin_fma(-l, u[c], x[c]);
            }
        } else if (finfo == 0) {
            finfo = jn + S + 1;
        }
        if constexpr (S + 1 < NB) r = 1.0 / x[S + 1];
    };
    // step S in the other waves: pivot row S from LDS
    auto step_wk = [&]<int S>() __attribute__((always_inline)) {
        if (S >= nbn) return;
        const double *us = sU + S * LDU;
        const double piv = us[S];
        const int km = min(kl, n - 1 - (jn + S));
        const int tt = t - S;
        const bool cand = own & (tt >= 1) & (tt <= km);
        viol |= cand && pivot_key(x[S], tt) > pivot_key(piv, 0);
        if (piv != 0.0) {
            double l;
            if (fabs(piv) >= DBL_MIN) {
                l = x[S] * us[NB];
            } else {
                l = x[S] / piv;
            }
            if (cand) {
                x[S] = l;
#pragma unroll
                for (int c = S + 1; c < NB; ++c) x[c] = __builtin_fma(-l, us[c], x[c]);
            }
        } else if (finfo == 0) {
            finfo = jn + S + 1;
        }
    };
    auto group_w0 = [&]<int G>() __attribute__((always_inline)) {
        if (G >= ngrp) return;
        [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
            (step_w0.template operator()<8 * G + Q>(), ...);
        }(std::make_integer_sequence<int, 8>{});
        // rows 8G..8G+7 are final: publish them with their reciprocals
        if (lane >= 8 * G && lane < 8 * G + 8) {
#pragma unroll
            for (int c = 8 * G; c < NB; ++c) sU[lane * LDU + c] = x[c];
            sU[lane * LDU + NB] = myrcp;
        }
        lds_barrier();
    };
    auto group_wk = [&]<int G>() __attribute__((always_inline)) {
        if (G >= ngrp) return;
        lds_barrier();
        [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
            (step_wk.template operator()<8 * G + Q>(), ...);
        }(std::make_integer_sequence<int, 8>{});
    };
    static_assert(NB == 32, "four groups of eight steps");
    if (__builtin_amdgcn_readfirstlane(wv) == 0) {  // (uniform, so each wave sees only its own barriers)
        group_w0.template operator()<0>();
        group_w0.template operator()<1>();
        group_w0.template operator()<2>();
        group_w0.template operator()<3>();
    } else {
        group_wk.template operator()<0>();
        group_wk.template operator()<1>();
        group_wk.template operator()<2>();
        group_wk.template operator()<3>();
    }
    if (__ballot(viol) && lane == 0) s_viol = 1;
    lds_barrier();
    bool verified = false;
    if (s_viol == 0) {
        // no interchange: pivots, multipliers and U entries stay in place
        if (t < nbn) ipiv[jn + t] = jn + t + 1;
        const int64_t st = colstep();
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            const int d = t - c;
            if (own && c < nbn && d >= -kv && d <= kl) AB[diag0 + c * st] = x[c];
        }
        if (t == 0 && finfo != 0 && P.info[bm] == 0) P.info[bm] = finfo;
        verified = true;
    }
    if (verified) return;
    load_panel();
    int myrow = t;
    int info = 0;
#pragma unroll 1
    for (int g = 0; g < NB / 8; ++g) {
        const int base = 8 * g;
        if (base >= nbn) break;
        // per step of the group: the row number this thread had once the
        // step's interchange was made, whether it then held a multiplier, and
        // (thread q) the pivot of step q; all stored when the group ends
        int rowat[8];
        unsigned lmask = 0;
        int mypiv = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int jj = base + q;
            if (jj < nbn) {
                const int col = jn + jj;
                const int km = min(kl, n - 1 - col);
                const int tt = myrow - jj;
                const bool cand = own & (tt >= 0) & (tt <= km);
                const double key = cand ? pivot_key(x[q], tt) : -2.0;
                const double wmax = wave_max_d(key);
                const bool top = key == wmax;
                unsigned long long hit = __ballot(top);
                if (__popcll(hit) > 1) {
                    // equal keys: the smallest row number wins (BLAS i_amax order)
                    const int mr = wave_min_i32(top ? myrow : INT_MAX);
                    hit = __ballot(top & (myrow == mr));
                }
                const int f = __builtin_amdgcn_readfirstlane(__builtin_ctzll(hit));
                // the wave's candidate, its reciprocal formed before the barrier
                const double cv = readlane_d(x[q], f);
                const double crcp = 1.0 / cv;
                const int crow = __builtin_amdgcn_readlane(cand ? myrow : INT_MAX, f);
                const int par = q & 1;
                if (lane == f) {
#pragma unroll
                    for (int c = q; c < NB; ++c) sW[par][wv][c] = x[c];
                    sK[par][wv] = wmax;
                    sR[par][wv] = crcp;
                    sI[par][wv] = crow;
                }
                lds_barrier();
                // best over the waves, without branches
                double bk = sK[par][0];
                int bi = sI[par][0], bw = 0;
#pragma unroll
                for (int w = 1; w < kWaves; ++w) {
                    const double kw = sK[par][w];
                    const int iw = sI[par][w];
                    const bool b = key_better(kw, iw, bk, bi);
                    bk = b ? kw : bk;
                    bi = b ? iw : bi;
                    bw = b ? w : bw;
                }
                bw = __builtin_amdgcn_readfirstlane(bw);
                bi = __builtin_amdgcn_readfirstlane(bi);
                const double *wr = sW[par][bw];
                const double piv = wr[q];
                const int p = bi - jj;
                mypiv = lane == q ? col + p + 1 : mypiv;
                const bool elim = piv != 0.0;  // uniform
                info = (!elim && info == 0) ? col + 1 : info;
                // interchange by renumbering (none for a zero pivot)
                const bool swp = elim & (p != 0);
                myrow = swp ? (myrow == bi ? jj : (myrow == jj ? bi : myrow)) : myrow;
                rowat[q] = myrow;
                const int tr = myrow - jj;
                const bool mrow = own & (tr >= 1) & (tr <= km);
                lmask |= unsigned(mrow) << q;
                double l;
                if (fabs(piv) >= DBL_MIN) {
                    l = x[q] * sR[par][bw];
                } else {
                    l = x[q] / piv;
                }
                // rows that are not eliminated get l = 0: fma(-0, u, x) leaves a
                // finite x as it is, up to the sign of a zero
                const double le = (mrow & elim) ? l : 0.0;
                x[q] = (mrow & elim) ? l : x[q];
#pragma unroll
                for (int c = q + 1; c < NB; ++c) x[c] = __builtin_fma(-le, wr[c], x[c]);
            }
        }
        // the group's pivots, multipliers (product form: each in the row it had
        // when its column was eliminated; for a zero pivot the entry as it is)
        // and finished rows of U; then the register row moves down eight columns
        if (t < 8 && base + t < nbn) ipiv[jn + base + t] = mypiv;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int jj = base + c;
            if ((lmask >> c) & 1u) AB[int64_t(jn + jj) * ldab + (kv + rowat[c] - jj)] = x[c];
        }
        if (myrow < nbn) {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int jj = base + c;
                const int d = myrow - jj;
                if (jj < nbn && d <= 0 && d >= -kv) AB[int64_t(jn + jj) * ldab + (kv + d)] = x[c];
            }
        }
#pragma unroll
        for (int c = 0; c < NB - 8; ++c) x[c] = x[c + 8];
#pragma unroll
        for (int c = NB - 8; c < NB; ++c) x[c] = 0.0;
    }
    if (t == 0 && info != 0 && P.info[bm] == 0) P.info[bm] = info;
}

}  // namespace

int launch_getrf_mfma(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s) {
    if (kl > kMaxKl || batch > 65535) {
        set_error("band_getrf: the matrix-core variant needs kl <= %d and batch <= 65535", kMaxKl);
        return BANDLU_ERR_UNSUPPORTED;
    }
    if (int rc = launch_band_zero_fill(n, kl, ku, dAB, ldab, strideAB, d_info, batch, s)) return rc;
    MfmaParams Q;
    Q.AB = dAB;
    Q.ipiv = d_ipiv;
    Q.info = d_info;
    Q.ldab = ldab;
    Q.strideAB = strideAB;
    Q.strideP = strideP;
    Q.n = (int)n;
    Q.kl = (int)kl;
    Q.ku = (int)ku;
    const int64_t kv = kl + ku;
    // launch k applies panel k-1 to the band it reaches and factors panel k
    for (int64_t jn = 0; jn < n; jn += NB) {
        Q.jn = (int)jn;
        Q.has_update = jn > 0;
        Q.j = (int)(jn - NB);
        int64_t blocks = 1;
        if (jn > 0) {
            const int64_t cend = std::min<int64_t>(n, jn + kv);  // panel k-1 reaches columns < j+NB+kv
            blocks = std::max<int64_t>(1, (cend - jn + NB - 1) / NB);
        }
        hipLaunchKernelGGL(mfma_step_kernel, dim3((unsigned)blocks, (unsigned)batch), dim3(kThreads),
                           0, s, Q);
        BANDLU_CHECK_LAUNCH("band_getrf (matrix-core step)");
    }
    return BANDLU_OK;
}

}  // namespace bandlu
