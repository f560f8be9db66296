// Step 3 of the structure-aware strategy (Sec. II-A cost f(N); Sec. III-A
// banded LU, xGBTRF): kernel selection and the unblocked any-bandwidth kernel.
//
// Variants (band_getrf_variant):
//   WINDOW      kl <= 31 and 2kl+ku+1 <= 64, or kl <= 15 and 2kl+ku+1 <= 128:
//               register window, 64 lanes per matrix (getrf_win64.hpp);
//   DIAG        1 <= kl, 1 <= ku <= 24, ldab <= 64 and kl small enough
//               for one lane per live row: every column is first factored
//               with its diagonal pivot and checked against partial pivoting
//               (getrf_diag.hpp); from the first column that fails, SPLIT
//               factors the rest;
//   SPLIT       1 <= kl <= 31 with the WINDOW limits: the window plus a
//               second wavefront that runs the pivot decisions
//               (getrf_split.hpp);
//   WINDOW_G16  batched, kl <= 7 and 2kl+ku+1 <= 32, or any batch with
//               1 <= kl <= 4 and 2kl+ku+1 <= 16: register window, 16 lanes
//               per matrix, four matrices per wavefront;
//   BLOCKED     kl <= 31 beyond the windows: panels of 32 columns factored in
//               registers, trailing band updated by many workgroups with the
//               unblocked rank-1 order (getrf_blocked.hip);
//   WIDE        32 <= kl <= 256 when the batch fits one launch of co-resident
//               workgroups: one persistent launch, blocks of 32 columns kept
//               in LDS, each panel factored by its block's owner and applied
//               by the others on the fp64 matrix cores (getrf_wide.hip);
//   BLOCKED_MFMA  32 <= kl <= 256 otherwise: one launch per panel, trailing
//               band updated as a dense product on the matrix cores
//               (getrf_mfma.hip);
//   GENERIC     kl > 256: one workgroup per matrix works on the band in global
//               memory, one column step at a time.
// The window, blocked and generic kernels produce bitwise the factors of the
// unblocked algorithm on finite data; the matrix-core variant agrees to
// rounding.  band_getrf_ex runs a named variant.
#include <algorithm>
#include <cfloat>
#include <climits>
#include <mutex>

#include "bufio.hpp"
#include "getrf_diag.hpp"
#include "getrf_window.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c1_h1_8(int H);
WinKernel win_kernel_g64_c1_h9_16(int H);
WinKernel win_kernel_g64_c1_h17_24(int H);
WinKernel win_kernel_g64_c1_h25_32(int H);
WinKernel win_kernel_g64_c2_h1_8(int H);
WinKernel win_kernel_g64_c2_h9_16(int H);
WinKernel win_kernel_g16_c1_h1_8(int H);
WinKernel win_kernel_g16_c2_h1_8(int H);
WinKernel split_kernel_c1_h2_16(int H);
WinKernel split_kernel_c1_h17_32(int H);
WinKernel split_kernel_c2_h2_16(int H);

// two-wavefront kernel (getrf_split.hpp) for 2 <= H <= 32
WinKernel lean64_fwd_kernel_c1(int H);
WinKernel lean64_fwd_kernel_c2(int H);

WinKernel split_kernel(int CPL, int H) {
    if (CPL == 1) return H <= 16 ? split_kernel_c1_h2_16(H) : split_kernel_c1_h17_32(H);
    return split_kernel_c2_h2_16(H);
}

// diagonal-pivot kernel (getrf_diag.hpp) for 1 <= ku <= kDiagMaxKu
WinKernel diag_kernel(int KU) {
    if (KU >= 1 && KU <= 8) return diag_kernel_ku1_8(KU);
    if (KU >= 9 && KU <= 16) return diag_kernel_ku9_16(KU);
    if (KU >= 17 && KU <= 24) return diag_kernel_ku17_24(KU);
    return nullptr;
}

bool diag_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab) {
    return kl >= 1 && ku >= 1 && ku <= kDiagMaxKu && kl <= diag_max_kl((int)ku) &&
           2 * kl + ku + 1 <= 64 && ldab <= 64 && n >= 2 && ldab * n * 8 <= kMaxBufferBytes;
}

WinKernel win_kernel(int G, int CPL, int H) {
    if (G == 16) {
        if (H > 8) return nullptr;
        return CPL == 1 ? win_kernel_g16_c1_h1_8(H) : win_kernel_g16_c2_h1_8(H);
    }
    if (CPL == 1) {
        if (H <= 8) return win_kernel_g64_c1_h1_8(H);
        if (H <= 16) return win_kernel_g64_c1_h9_16(H);
        if (H <= 24) return win_kernel_g64_c1_h17_24(H);
        return win_kernel_g64_c1_h25_32(H);
    }
    if (H <= 8) return win_kernel_g64_c2_h1_8(H);
    if (H <= 16) return win_kernel_g64_c2_h9_16(H);
    return nullptr;
}

int launch_getrf_blocked(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                         int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                         int64_t batch, hipStream_t s);
int launch_getrf_mfma(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s);
int launch_getrf_wide(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s, void *ws, size_t ws_bytes,
                      double *dB = nullptr, int64_t ldb = 0, int64_t strideB = 0,
                      int64_t nrhs = 0);
bool getrf_wide_fits(int64_t n, int64_t kl, int64_t ku, int64_t batch);
bool getrf_wide_one_launch(int64_t n, int64_t kl, int64_t ku, int64_t batch);
size_t getrf_wide_scratch_bytes(int64_t n, int64_t kl, int64_t ku, int64_t batch);

namespace {

constexpr int kGenThreads = 256;

struct GenParams {
    double *AB;
    int32_t *ipiv;
    int32_t *info;
    int64_t n, kl, ku, ldab, strideAB, strideP;
    int64_t m;  // rows (m x n band matrix; m = n for the square factorisation)
};

// pivot key: |x|, with a NaN ranked first in position 0 and last elsewhere, so
// that (largest key, smallest index) equals the BLAS i_amax choice
__device__ inline double pivot_key(double x, int64_t t) {
    if (__builtin_isnan(x)) return t == 0 ? __builtin_inf() : -1.0;
    return fabs(x);
}

__device__ inline bool key_better(double ka, int64_t ia, double kb, int64_t ib) {
    return ka > kb || (ka == kb && ia < ib);
}

__global__ __launch_bounds__(kGenThreads) void getrf_generic_kernel(GenParams P) {
    const int64_t b = blockIdx.x;
    double *__restrict__ AB = P.AB + b * P.strideAB;
    int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    const int64_t n = P.n, m = P.m, kl = P.kl, ku = P.ku, kv = kl + ku, ldab = P.ldab;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    __shared__ double s_key[kGenThreads / 64];
    __shared__ int64_t s_idx[kGenThreads / 64];
    __shared__ int64_t s_p;
    __shared__ int s_nz;

    // in-matrix fill slots start at zero
    if (kl > 0) {
        // (columns by wavefront, fill rows by lane: no per-entry division)
        for (int64_t c = wv; c < n; c += kGenThreads / 64)
            for (int64_t r = lane; r < kl; r += 64)
                if (r >= kv - c && r - kv + c < m) AB[c * ldab + r] = 0.0;
    }
    __syncthreads();

    int64_t ju = 0;
    int32_t info = 0;
    const int64_t steps = min(m, n);
    for (int64_t j = 0; j < steps; ++j) {
        const int64_t km = min(kl, m - 1 - j);
        double *colj = AB + j * ldab + kv;  // colj[t] = a(j+t, j)
        double bk = -2.0;
        int64_t bi = INT64_MAX;
        for (int64_t t = tid; t <= km; t += kGenThreads) {
            const double k = pivot_key(colj[t], t);
            if (key_better(k, t, bk, bi)) { bk = k; bi = t; }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const double ok = __shfl_xor(bk, o, 64);
            const int64_t oi = __shfl_xor(bi, o, 64);
            if (key_better(ok, oi, bk, bi)) { bk = ok; bi = oi; }
        }
        if (lane == 0) { s_key[wv] = bk; s_idx[wv] = bi; }
        __syncthreads();
        if (tid == 0) {
            double kk = s_key[0];
            int64_t ii = s_idx[0];
            for (int w = 1; w < kGenThreads / 64; ++w)
                if (key_better(s_key[w], s_idx[w], kk, ii)) { kk = s_key[w]; ii = s_idx[w]; }
            s_p = ii;
            s_nz = colj[ii] != 0.0;
            ipiv[j] = int32_t(j + ii + 1);
        }
        __syncthreads();
        const int64_t p = s_p;
        if (s_nz) {
            ju = max(ju, min(j + ku + p, n - 1));
            if (p != 0) {
                for (int64_t c = j + tid; c <= ju; c += kGenThreads) {
                    double *x = AB + c * ldab + (kv + j - c);
                    const double t0 = x[0];
                    x[0] = x[p];
                    x[p] = t0;
                }
                __syncthreads();
            }
            const double piv = colj[0];
            if (fabs(piv) >= DBL_MIN) {
                const double rcp = 1.0 / piv;
                for (int64_t t = 1 + tid; t <= km; t += kGenThreads) colj[t] = colj[t] * rcp;
            } else {
                for (int64_t t = 1 + tid; t <= km; t += kGenThreads) colj[t] = colj[t] / piv;
            }
            __syncthreads();
            if (km > 0) {
                // columns j+1..ju by wavefront, rows by lane (no per-entry
                // index division; one column's entries are contiguous)
                constexpr int kGenWaves = kGenThreads / 64;
                for (int64_t c = j + 1 + wv; c <= ju; c += kGenWaves) {
                    double *x = AB + c * ldab + (kv + j - c);  // x[0] = a(j, c)
                    const double u = x[0];
                    for (int64_t t = 1 + lane; t <= km; t += 64)
                        x[t] = __builtin_fma(-colj[t], u, x[t]);
                }
            }
            __syncthreads();
        } else if (info == 0) {
            info = int32_t(j + 1);
        }
    }
    if (tid == 0) P.info[b] = info;
}

__global__ void zero_info_kernel(int32_t *info, int64_t batch) {
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < batch) info[i] = 0;
}

// Up to this kl the one-wavefront window kernel with wave-uniform pivots
// (getrf_lean64.hpp) takes fewer cycles per column than the two-wavefront
// kernel, for single matrices and after a failed diagonal-pivot check.
constexpr int64_t kLeanMaxKl = 6;

int select_variant(int64_t n, int64_t kl, int64_t ku, int64_t batch) {
    const int64_t need = 2 * kl + ku + 1;
    if (batch >= 64 && kl <= 7 && need <= 32) return BANDLU_GETRF_WINDOW_G16;
    // a few matrices with a very small band: the sixteen-lane kernel's step
    // does not depend on whether rows are interchanged, and for kl <= 4 it
    // is within about 10 % of DIAG when none are and 2x faster when they are
    if (kl >= 1 && kl <= 4 && need <= 16) return BANDLU_GETRF_WINDOW_G16;
    if (diag_fits(n, kl, ku, need)) return BANDLU_GETRF_DIAG;
    if (kl >= 1 && kl <= kLeanMaxKl && need <= 128 && need * n * 8 <= kMaxBufferBytes)
        return BANDLU_GETRF_WINDOW;
    if (kl >= 1 && kl <= 31 && (need <= 64 || (need <= 128 && kl <= 15)) &&
        need * n * 8 <= kMaxBufferBytes)
        return BANDLU_GETRF_SPLIT;
    if (kl <= 31 && (need <= 64 || (need <= 128 && kl <= 15)) && need * n * 8 <= kMaxBufferBytes)
        return BANDLU_GETRF_WINDOW;
    // from kl = 32 on, applying a panel of 32 columns is a real dense product
    // (at least 32 x 32 x 32): matrix cores, in one persistent launch when the
    // batch fits the co-resident workgroups, else one launch per panel
    if (kl >= 32 && kl <= 256 && getrf_wide_one_launch(n, kl, ku, batch))
        return BANDLU_GETRF_WIDE;
    if (kl <= 256 && n <= INT32_MAX && batch <= 65535)
        return kl >= 32 ? BANDLU_GETRF_BLOCKED_MFMA : BANDLU_GETRF_BLOCKED;
    return BANDLU_GETRF_GENERIC;
}

// Whether a variant can factor these sizes (the window kernels address the
// band through a range-checked buffer of at most 2 GiB and keep the window in
// registers; the blocked kernels hold a panel of NB + kl rows in one workgroup).
bool variant_fits(int v, int64_t n, int64_t kl, int64_t ku, int64_t ldab, int64_t batch) {
    const int64_t need = 2 * kl + ku + 1;
    switch (v) {
    case BANDLU_GETRF_WINDOW_G16:
        return kl <= 7 && need <= 32 && ldab * n * 8 <= kMaxBufferBytes;
    case BANDLU_GETRF_WINDOW:
        return kl <= 31 && (need <= 64 || (need <= 128 && kl <= 15)) &&
               ldab * n * 8 <= kMaxBufferBytes;
    case BANDLU_GETRF_SPLIT:
        return kl >= 1 && kl <= 31 && (need <= 64 || (need <= 128 && kl <= 15)) &&
               ldab * n * 8 <= kMaxBufferBytes;
    case BANDLU_GETRF_DIAG:
        return diag_fits(n, kl, ku, ldab);
    case BANDLU_GETRF_BLOCKED:
    case BANDLU_GETRF_BLOCKED_MFMA:
        return kl <= 256 && batch <= 65535;
    case BANDLU_GETRF_WIDE:
        return getrf_wide_fits(n, kl, ku, batch);
    case BANDLU_GETRF_GENERIC:
        return true;
    default:
        return false;
    }
}

// ws / ws_bytes: a caller's scratch buffer for the persistent wide-band
// kernel, or null to let it take one from the stream-ordered allocator (the
// other kernels need none)
int launch_getrf(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                 int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                 int64_t batch, int variant, hipStream_t s, void *ws = nullptr,
                 size_t ws_bytes = 0) {
    if (batch == 0) return BANDLU_OK;
    if (n == 0) {
        hipLaunchKernelGGL(zero_info_kernel, dim3((unsigned)((batch + 255) / 256)), dim3(256), 0,
                           s, d_info, batch);
        BANDLU_CHECK_LAUNCH("band_getrf (n = 0)");
        return BANDLU_OK;
    }
    const int64_t need = 2 * kl + ku + 1;
    int v = variant;
    if (v == 0) {
        v = select_variant(n, kl, ku, batch);
        if (!variant_fits(v, n, kl, ku, ldab, batch)) {
            // the caller's ldab (or stride) rules out the kernel chosen from the
            // sizes alone: take the next kernel in the order of preference that
            // fits, the one-workgroup kernel last
            const int chain[] = {BANDLU_GETRF_WINDOW_G16, BANDLU_GETRF_DIAG, BANDLU_GETRF_SPLIT,
                                 BANDLU_GETRF_WINDOW,
                                 kl >= 32 ? BANDLU_GETRF_BLOCKED_MFMA : BANDLU_GETRF_BLOCKED};
            int k = 0;
            while (k < 5 && chain[k] != v) ++k;
            v = BANDLU_GETRF_GENERIC;
            for (++k; k < 5; ++k)
                if (variant_fits(chain[k], n, kl, ku, ldab, batch)) { v = chain[k]; break; }
        }
    } else if (!variant_fits(v, n, kl, ku, ldab, batch)) {
        set_error("band_getrf: variant %d cannot factor n = %lld, kl = %lld, ku = %lld", v,
                  (long long)n, (long long)kl, (long long)ku);
        return BANDLU_ERR_UNSUPPORTED;
    }
    if (v == BANDLU_GETRF_WINDOW || v == BANDLU_GETRF_WINDOW_G16) {
        WinParams W;
        W.AB = dAB;
        W.ipiv = d_ipiv;
        W.info = d_info;
        W.ldab = ldab;
        W.strideAB = strideAB;
        W.strideP = strideP;
        W.n = (int)n;
        W.ku = (int)ku;
        W.batch = (int)batch;
        W.kl = (int)kl;
        W.resume = 0;
        const int H = (int)kl + 1;
        WinKernel k;
        int per_wave;
        if (v == BANDLU_GETRF_WINDOW_G16) {
            // one column per lane addresses the whole batch through one
            // range-checked buffer: it must stay below 2 GiB
            const bool one = need <= 16 && batch * strideAB * 8 <= kMaxBufferBytes &&
                             batch * strideP * 4 <= kMaxBufferBytes;
            k = win_kernel(16, one ? 1 : 2, H);
            per_wave = 4;
        } else {
            k = win_kernel(64, need <= 64 ? 1 : 2, H);
            per_wave = 1;
        }
        if (!k) {
            set_error("band_getrf: no window kernel for kl = %lld", (long long)kl);
            return BANDLU_ERR_UNSUPPORTED;
        }
        const int64_t blocks = (batch + per_wave - 1) / per_wave;
        hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(64), 0, s, W);
        BANDLU_CHECK_LAUNCH("band_getrf (window)");
        return BANDLU_OK;
    }
    if (v == BANDLU_GETRF_SPLIT) {
        WinParams W;
        W.AB = dAB;
        W.ipiv = d_ipiv;
        W.info = d_info;
        W.ldab = ldab;
        W.strideAB = strideAB;
        W.strideP = strideP;
        W.n = (int)n;
        W.ku = (int)ku;
        W.batch = (int)batch;
        W.kl = (int)kl;
        W.resume = 0;
        const WinKernel k = split_kernel(need <= 64 ? 1 : 2, (int)kl + 1);
        if (!k) {
            set_error("band_getrf: no two-wavefront kernel for kl = %lld", (long long)kl);
            return BANDLU_ERR_UNSUPPORTED;
        }
        hipLaunchKernelGGL(k, dim3((unsigned)batch), dim3(128), 0, s, W);
        BANDLU_CHECK_LAUNCH("band_getrf (two wavefronts)");
        return BANDLU_OK;
    }
    if (v == BANDLU_GETRF_DIAG) {
        WinParams W;
        W.AB = dAB;
        W.ipiv = d_ipiv;
        W.info = d_info;
        W.ldab = ldab;
        W.strideAB = strideAB;
        W.strideP = strideP;
        W.n = (int)n;
        W.ku = (int)ku;
        W.batch = (int)batch;
        W.kl = (int)kl;
        W.resume = 0;
        const WinKernel k = diag_kernel((int)ku);
        // (the band fits 64 lanes: 2kl+ku+1 <= 64)
        const bool lean = kl <= kLeanMaxKl;
        const WinKernel rest = lean ? win_kernel(64, 1, (int)kl + 1) : split_kernel(1, (int)kl + 1);
        if (!k || !rest) {
            set_error("band_getrf: no diagonal-pivot kernel for kl = %lld, ku = %lld", (long long)kl,
                      (long long)ku);
            return BANDLU_ERR_UNSUPPORTED;
        }
        hipLaunchKernelGGL(k, dim3((unsigned)batch), dim3(64), 0, s, W);
        BANDLU_CHECK_LAUNCH("band_getrf (diagonal pivots)");
        // columns from the first failing one on (a launch that returns at
        // once where every column passed)
        W.resume = 1;
        hipLaunchKernelGGL(rest, dim3((unsigned)batch), dim3(lean ? 64 : 128), 0, s, W);
        BANDLU_CHECK_LAUNCH("band_getrf (diagonal pivots, resumed)");
        return BANDLU_OK;
    }
    if (v == BANDLU_GETRF_BLOCKED)
        return launch_getrf_blocked(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch,
                                    s);
    if (v == BANDLU_GETRF_BLOCKED_MFMA)
        return launch_getrf_mfma(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch, s);
    if (v == BANDLU_GETRF_WIDE)
        return launch_getrf_wide(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch, s,
                                 ws, ws_bytes);
    GenParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.info = d_info;
    P.n = n;
    P.m = n;
    P.kl = kl;
    P.ku = ku;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    hipLaunchKernelGGL(getrf_generic_kernel, dim3((unsigned)batch), dim3(kGenThreads), 0, s, P);
    BANDLU_CHECK_LAUNCH("band_getrf (generic)");
    return BANDLU_OK;
}

}  // namespace

// band_gbsv_lu for one right-hand side where the lean window kernel is the
// one band_getrf runs: the factorisation and the forward solve in one launch.
// Returns BANDLU_ERR_UNSUPPORTED (having launched nothing) where it is not.
int launch_getrf_lean_fwd(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int32_t *d_ipiv, double *dB, int32_t *d_info, hipStream_t s) {
    const int64_t need = 2 * kl + ku + 1;
    if (n < 1 || kl < 1 || kl > kLeanMaxKl || select_variant(n, kl, ku, 1) != BANDLU_GETRF_WINDOW ||
        !variant_fits(BANDLU_GETRF_WINDOW, n, kl, ku, ldab, 1) || n * 8 > kMaxBufferBytes)
        return BANDLU_ERR_UNSUPPORTED;
    const int H = (int)kl + 1;
    const WinKernel k = need <= 64 ? lean64_fwd_kernel_c1(H) : lean64_fwd_kernel_c2(H);
    if (!k) return BANDLU_ERR_UNSUPPORTED;
    WinParams W;
    W.AB = dAB;
    W.ipiv = d_ipiv;
    W.info = d_info;
    W.ldab = ldab;
    W.strideAB = ldab * n;
    W.strideP = n;
    W.n = (int)n;
    W.ku = (int)ku;
    W.batch = 1;
    W.kl = (int)kl;
    W.resume = 0;
    W.B = dB;
    W.strideB = n;
    hipLaunchKernelGGL(k, dim3(1), dim3(64), 0, s, W);
    BANDLU_CHECK_LAUNCH("band_gbsv_lu (lean window with the forward solve)");
    return BANDLU_OK;
}

}  // namespace bandlu

using namespace bandlu;

extern "C" int band_getrf_variant(int64_t n, int64_t kl, int64_t ku, int64_t batch) {
    const int64_t bmax = n > 1 ? n - 1 : 0;
    if (n < 0) return -1;
    if (kl < 0 || kl > bmax) return -2;
    if (ku < 0 || ku > bmax) return -3;
    if (batch < 0) return -4;
    return select_variant(n, kl, ku, batch);
}

extern "C" int band_getrf(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int32_t *d_ipiv, int32_t *d_info, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrf: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrf: kl out of [0, max(0, n-1)]");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrf: ku out of [0, max(0, n-1)]");
    BANDLU_ARG(n == 0 || dAB != nullptr, 4, "band_getrf: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 5, "band_getrf: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || d_ipiv != nullptr, 6, "band_getrf: d_ipiv is null");
    BANDLU_ARG(d_info != nullptr, 7, "band_getrf: d_info is null");
    if (n > kMaxN) {
        set_error("band_getrf: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrf(n, kl, ku, dAB, ldab, ldab * n, d_ipiv, n, d_info, 1, 0, as_stream(stream));
}

extern "C" int band_getrf_batched(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                                  int64_t strideAB, int32_t *d_ipiv, int64_t strideP,
                                  int32_t *d_info, int64_t batch, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrf_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrf_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrf_batched: ku out of range");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 4, "band_getrf_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 5, "band_getrf_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 6, "band_getrf_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 7, "band_getrf_batched: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 8, "band_getrf_batched: strideP < n");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 9, "band_getrf_batched: d_info is null");
    BANDLU_ARG(batch >= 0, 10, "band_getrf_batched: batch < 0");
    if (n > kMaxN || batch > INT_MAX) {
        set_error("band_getrf_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrf(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch, 0,
                        as_stream(stream));
}

extern "C" int band_getrf_ex(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                             int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                             int64_t batch, int variant, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrf_ex: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrf_ex: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrf_ex: ku out of range");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 4, "band_getrf_ex: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 5, "band_getrf_ex: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 6, "band_getrf_ex: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 7, "band_getrf_ex: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 8, "band_getrf_ex: strideP < n");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 9, "band_getrf_ex: d_info is null");
    BANDLU_ARG(batch >= 0, 10, "band_getrf_ex: batch < 0");
    BANDLU_ARG(variant >= 0 && variant <= BANDLU_GETRF_WIDE, 11,
               "band_getrf_ex: unknown variant");
    if (n > kMaxN || batch > INT_MAX) {
        set_error("band_getrf_ex: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrf(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch, variant,
                        as_stream(stream));
}

// ------------------------------------------------- no-allocation entry --
// The persistent wide-band kernel's hand-off ring (counters and published
// panels) lives in a fixed device array instead of stream-ordered memory, so
// that a caller that cannot allocate can factor any band the library would
// factor with it, up to kNoAllocScratchBytes of ring per matrix.  Every
// device the entry point runs on holds its own copy of the array until the
// process ends; host code reaches it only through the address looked up once
// per device (the array's name is a host-side stand-in, not a device address).
namespace bandlu {
namespace {
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
constexpr int kNoAllocMaxDevices = 64;
std::mutex g_noalloc_mu;
void *g_noalloc_ptr[kNoAllocMaxDevices];
}  // namespace
}  // namespace bandlu

static __device__ __align__(256) char scratch[bandlu::kNoAllocScratchBytes];

// device address of `scratch` on the current device
static int noalloc_scratch(void **out) {
    int dev = -1;
    if (hipError_t e = hipGetDevice(&dev); e != hipSuccess)
        return hip_fail(e, "band_getrf_batched_noalloc (current device)");
    if (dev < 0 || dev >= kNoAllocMaxDevices) {
        set_error("band_getrf_batched_noalloc: device %d beyond the %d the library tracks", dev,
                  kNoAllocMaxDevices);
        return BANDLU_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    if (g_noalloc_ptr[dev] == nullptr) {
        void *p = nullptr;
        if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess)
            return hip_fail(e, "band_getrf_batched_noalloc (scratch address)");
        g_noalloc_ptr[dev] = p;
    }
    *out = g_noalloc_ptr[dev];
    return BANDLU_OK;
}

extern "C" int band_getrf_batched_noalloc(int64_t n, int64_t kl, int64_t ku, double *dAB,
                                          int64_t ldab, int64_t strideAB, int32_t *d_ipiv,
                                          int64_t strideP, int32_t *d_info, int64_t batch,
                                          void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrf_batched_noalloc: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrf_batched_noalloc: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrf_batched_noalloc: ku out of range");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 4, "band_getrf_batched_noalloc: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 5, "band_getrf_batched_noalloc: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 6,
               "band_getrf_batched_noalloc: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 7,
               "band_getrf_batched_noalloc: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 8, "band_getrf_batched_noalloc: strideP < n");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 9, "band_getrf_batched_noalloc: d_info is null");
    BANDLU_ARG(batch >= 0, 10, "band_getrf_batched_noalloc: batch < 0");
    if (n > kMaxN || batch > INT_MAX) {
        set_error("band_getrf_batched_noalloc: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    // the kernel band_getrf_batched would take; only the persistent wide-band
    // one needs scratch, and it gets the fixed array
    void *ws = nullptr;
    size_t ws_bytes = 0;
    if (n > 0 && batch > 0 && select_variant(n, kl, ku, batch) == BANDLU_GETRF_WIDE) {
        const size_t per = getrf_wide_scratch_bytes(n, kl, ku, 1);
        if (per > kNoAllocScratchBytes) {
            set_error("band_getrf_batched_noalloc: kl = %lld, ku = %lld needs %zu bytes of "
                      "scratch per matrix, beyond the %zu this entry point holds per device",
                      (long long)kl, (long long)ku, per, kNoAllocScratchBytes);
            return BANDLU_ERR_UNSUPPORTED;
        }
        if (int rc = noalloc_scratch(&ws); rc != BANDLU_OK) return rc;
        ws_bytes = kNoAllocScratchBytes;
    }
    return launch_getrf(n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch, 0,
                        as_stream(stream), ws, ws_bytes);
}

// ------------------------------------------------- rectangular m x n --
// The band LU of an m x n band matrix (xGBTRF with m != n): the one-workgroup
// kernel above with m rows, min(m, n) column steps and km = min(kl, m-1-j)
// candidates per step; element (i, j), 0 <= i < m, at AB[kl+ku+i-j + j*ldab].
namespace bandlu {
namespace {
int getrf_mn(int64_t m, int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
             int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info, int64_t batch,
             hipStream_t s) {
    if (batch == 0) return BANDLU_OK;
    GenParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.info = d_info;
    P.n = n;
    P.m = m;
    P.kl = kl;
    P.ku = ku;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    hipLaunchKernelGGL(getrf_generic_kernel, dim3((unsigned)batch), dim3(kGenThreads), 0, s, P);
    BANDLU_CHECK_LAUNCH("band_getrf_mn");
    return BANDLU_OK;
}
}  // namespace
}  // namespace bandlu

extern "C" int band_getrf_mn(int64_t m, int64_t n, int64_t kl, int64_t ku, double *dAB,
                             int64_t ldab, int32_t *d_ipiv, int32_t *d_info, void *stream) {
    clear_error();
    BANDLU_ARG(m >= 0, 1, "band_getrf_mn: m < 0");
    BANDLU_ARG(n >= 0, 2, "band_getrf_mn: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= (m > 1 ? m - 1 : 0), 3, "band_getrf_mn: kl out of [0, max(0, m-1)]");
    BANDLU_ARG(ku >= 0 && ku <= (n > 1 ? n - 1 : 0), 4, "band_getrf_mn: ku out of [0, max(0, n-1)]");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_getrf_mn: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrf_mn: ldab < 2kl+ku+1");
    BANDLU_ARG(m == 0 || n == 0 || d_ipiv != nullptr, 7, "band_getrf_mn: d_ipiv is null");
    BANDLU_ARG(d_info != nullptr, 8, "band_getrf_mn: d_info is null");
    if (m > kMaxN || n > kMaxN) {
        set_error("band_getrf_mn: sizes >= 2^31 are not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return getrf_mn(m, n, kl, ku, dAB, ldab, ldab * n, d_ipiv, std::min(m, n), d_info, 1,
                    as_stream(stream));
}

extern "C" int band_getrf_mn_batched(int64_t m, int64_t n, int64_t kl, int64_t ku, double *dAB,
                                     int64_t ldab, int64_t strideAB, int32_t *d_ipiv,
                                     int64_t strideP, int32_t *d_info, int64_t batch,
                                     void *stream) {
    clear_error();
    BANDLU_ARG(m >= 0, 1, "band_getrf_mn_batched: m < 0");
    BANDLU_ARG(n >= 0, 2, "band_getrf_mn_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= (m > 1 ? m - 1 : 0), 3, "band_getrf_mn_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= (n > 1 ? n - 1 : 0), 4, "band_getrf_mn_batched: ku out of range");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_getrf_mn_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrf_mn_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_getrf_mn_batched: strideAB < ldab*n");
    BANDLU_ARG(m == 0 || n == 0 || batch == 0 || d_ipiv != nullptr, 8,
               "band_getrf_mn_batched: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= std::min(m, n), 9,
               "band_getrf_mn_batched: strideP < min(m, n)");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 10, "band_getrf_mn_batched: d_info is null");
    BANDLU_ARG(batch >= 0, 11, "band_getrf_mn_batched: batch < 0");
    if (m > kMaxN || n > kMaxN || batch > 65535) {
        set_error("band_getrf_mn_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return getrf_mn(m, n, kl, ku, dAB, ldab, strideAB, d_ipiv, strideP, d_info, batch,
                    as_stream(stream));
}
