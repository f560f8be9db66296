// Band Cholesky for symmetric positive definite bands: the Cholesky case the
// paper names beside LU (end of Sec. II-B), on the symmetric structure that
// the first step of Sec. II-A looks for.
//
//  * band_is_symmetric: A(i,j) == A(j,i) for 0 < i-j <= kd, read from the
//    dense matrix (IEEE comparison: -0.0 matches +0.0, NaN matches nothing).
//  * band_pbtrf: A = L L^T, lower band in LAPACK's layout (element (i, j),
//    j <= i <= j+kd, at AB[i - j + j*ldab]).  One workgroup per matrix,
//    right-looking: step j takes d = sqrt(A(j,j)) (stops with info = j+1 when
//    A(j,j) is not > 0), scales column j by r = 1/d and applies
//    A(i,c) -= L(i,j) L(c,j) to the trailing kd x kd triangle, one fused
//    multiply-add per entry and step in the order of the steps, so the factor
//    is bitwise that of the unblocked definition.  For kd <= 140 the columns
//    j..j+kd+1 live in LDS (kd+2 column slots, so the column that enters is
//    written while the step reads the others: one barrier per step); wider
//    bands are updated in place in global memory.
//  * band_pbtrs: L y = b forward and L^T x = y backward, the dividing forward
//    chain over L's columns and the backward chain over its rows.
#include <algorithm>
#include <climits>

#include "getrs_ring.hpp"

namespace bandlu {

int launch_chain(int mode, const RingParams &P, int64_t batch, hipStream_t s);

namespace {

constexpr int kCholThreads = 256;
constexpr int kCholLdsMaxKd = 140;

struct CholParams {
    double *AB;
    int32_t *info;
    int64_t ldab, strideAB;
    int n, kd;
};

// LDS window: column c at slot c % (kd+2), entry r (row c+r) at slot*(kd+1)+r
__global__ __launch_bounds__(kCholThreads) void pbtrf_lds_kernel(CholParams P) {
    extern __shared__ double win[];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int n = P.n, kd = P.kd, W = kd + 2, H = kd + 1;
    double *AB = P.AB + int64_t(blockIdx.x) * P.strideAB;
    const int64_t ldab = P.ldab;
    auto at = [&](int c, int r) -> double & { return win[(c % W) * H + r]; };
    // columns 0..kd enter
    for (int q = tid; q < (kd + 1) * H; q += kCholThreads) {
        const int c = q / H, r = q - c * H;
        if (c < n) at(c, r) = c + r < n ? AB[r + int64_t(c) * ldab] : 0.0;
    }
    __syncthreads();
    int info = 0;
    // the columns that enter are read kPf steps ahead (a register ring), so
    // that no step waits for its load
    constexpr int kPf = 4;
    auto ld_enter = [&](int ce) -> double {
        return (ce < n && tid < H && ce + tid < n) ? AB[tid + int64_t(ce) * ldab] : 0.0;
    };
    double ring[kPf];
#pragma unroll
    for (int q = 0; q < kPf; ++q) ring[q] = ld_enter(kd + 1 + q);
    for (int j0 = 0; j0 < n && !info; j0 += kPf)
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
        const int j = j0 + q;
        if (j >= n) break;
        const int kn = std::min(kd, n - 1 - j);
        // the column that enters (j+kd+1), loaded kPf steps ago
        const int ce = j + kd + 1;
        const double enter = ring[q];
        ring[q] = ld_enter(ce + kPf);
        const double d0 = at(j, 0);
        if (!(d0 > 0.0)) {
            info = j + 1;
            break;
        }
        const double d = __builtin_sqrt(d0);
        const double r = 1.0 / d;
        // trailing update A(j+b, j+a) for 1 <= a <= b <= kn: column j+a by
        // wavefront, rows by lane (L(., j) formed where it is used)
        const int sj = j % W;  // (one modulo per step; the other slots follow from it)
        const double *cj = win + sj * H;
        for (int a = 1 + wv; a <= kn; a += kCholThreads / 64) {
            const int sa = sj + a >= W ? sj + a - W : sj + a;
            double *ca = win + sa * H;
            const double la = cj[a] * r;
            for (int b = a + lane; b <= kn; b += 64)
                ca[b - a] = __builtin_fma(-(cj[b] * r), la, ca[b - a]);
        }
        // column j is final
        if (tid <= kn) AB[tid + int64_t(j) * ldab] = tid == 0 ? d : cj[tid] * r;
        if (ce < n && tid < H) at(ce, tid) = enter;
        __syncthreads();
    }
    if (info) {
        // not positive definite at column info-1: the window's columns keep
        // their updated values, as the unblocked algorithm leaves them
        const int j = info - 1;
        for (int q = tid; q < (kd + 1) * H; q += kCholThreads) {
            const int c = j + q / H, r = q % H;
            if (c < n && c + r < n && c <= j + kd) AB[r + int64_t(c) * ldab] = at(c, r);
        }
    }
    if (tid == 0) P.info[blockIdx.x] = info;
}

__global__ __launch_bounds__(kCholThreads) void pbtrf_global_kernel(CholParams P) {
    const int tid = threadIdx.x;
    const int n = P.n, kd = P.kd;
    double *AB = P.AB + int64_t(blockIdx.x) * P.strideAB;
    const int64_t ldab = P.ldab;
    auto at = [&](int c, int r) -> double & { return AB[r + int64_t(c) * ldab]; };
    int info = 0;
    for (int j = 0; j < n; ++j) {
        const int kn = std::min(kd, n - 1 - j);
        const double d0 = at(j, 0);
        if (!(d0 > 0.0)) {
            info = j + 1;
            break;
        }
        const double d = __builtin_sqrt(d0);
        const double r = 1.0 / d;
        // column j+a by wavefront, rows by lane
        const int wvg = tid >> 6, lng = tid & 63;
        for (int a = 1 + wvg; a <= kn; a += kCholThreads / 64) {
            const double la = at(j, a) * r;
            for (int b = a + lng; b <= kn; b += 64)
                at(j + a, b - a) = __builtin_fma(-(at(j, b) * r), la, at(j + a, b - a));
        }
        __syncthreads();
        // column j is final (no later step reads it)
        for (int t = tid; t <= kn; t += kCholThreads) at(j, t) = t == 0 ? d : at(j, t) * r;
    }
    if (tid == 0) P.info[blockIdx.x] = info;
}

__global__ void sym_init_kernel(int32_t *flag) { *flag = 1; }

__global__ void sym_check_kernel(const double *A, int64_t n, int64_t lda, int64_t kd,
                                 int32_t *flag) {
    const int64_t total = n * kd;
    for (int64_t g = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; g < total;
         g += int64_t(gridDim.x) * blockDim.x) {
        const int64_t j = g / kd, d = g - j * kd + 1;
        if (j + d < n && !(A[j + d + j * lda] == A[j + (j + d) * lda])) *flag = 0;
    }
}

int pbtrf(int64_t n, int64_t kd, double *dAB, int64_t ldab, int64_t strideAB, int32_t *d_info,
          int64_t batch, hipStream_t s) {
    if (batch == 0) return BANDLU_OK;
    CholParams P;
    P.AB = dAB;
    P.info = d_info;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.n = (int)n;
    P.kd = (int)kd;
    if (kd <= kCholLdsMaxKd) {
        const size_t shm = size_t(kd + 2) * size_t(kd + 1) * sizeof(double);
        if (shm > 64 * 1024) {
            if (hipError_t e = hipFuncSetAttribute((const void *)pbtrf_lds_kernel,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                                   (int)shm);
                e != hipSuccess)
                return hip_fail(e, "band_pbtrf (LDS window size)");
        }
        hipLaunchKernelGGL(pbtrf_lds_kernel, dim3((unsigned)batch), dim3(kCholThreads), shm, s, P);
    } else {
        hipLaunchKernelGGL(pbtrf_global_kernel, dim3((unsigned)batch), dim3(kCholThreads), 0, s,
                           P);
    }
    BANDLU_CHECK_LAUNCH("band_pbtrf");
    return BANDLU_OK;
}

int pbtrs(int64_t n, int64_t kd, int64_t nrhs, const double *dAB, int64_t ldab, int64_t strideAB,
          double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    RingParams P{};
    P.AB = dAB;
    P.B = dB;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.ldb = ldb;
    P.strideB = strideB;
    P.n = (int)n;
    P.nrhs = (int)nrhs;
    P.nsteps = (int)n;
    P.K = (int)kd;
    // L y = b: column j from its diagonal (row 0 of the lower layout) down
    P.cb0 = 0;
    P.es = 1;
    if (int rc = launch_chain(kRingFwdDiv, P, batch, s); rc != BANDLU_OK) return rc;
    // L^T x = y: step j is column n-1-j of L^T, i.e. row col of L; entry e is
    // L(col, col-kd+e) at (kd-e) + (col-kd+e)*ldab
    P.cb0 = kd * (1 - ldab);
    P.es = ldab - 1;
    return launch_chain(kRingBwd, P, batch, s);
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int band_is_symmetric(const double *dA, int64_t n, int64_t lda, int64_t kd,
                                 int32_t *d_flag, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 2, "band_is_symmetric: n < 0");
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "band_is_symmetric: lda < max(1, n)");
    BANDLU_ARG(kd >= 0 && kd <= (n > 1 ? n - 1 : 0), 4, "band_is_symmetric: kd out of range");
    BANDLU_ARG(n == 0 || dA != nullptr, 1, "band_is_symmetric: dA is null");
    BANDLU_ARG(d_flag != nullptr, 5, "band_is_symmetric: d_flag is null");
    hipStream_t s = as_stream(stream);
    hipLaunchKernelGGL(sym_init_kernel, dim3(1), dim3(1), 0, s, d_flag);
    BANDLU_CHECK_LAUNCH("band_is_symmetric (init)");
    if (n > 1 && kd > 0) {
        const int64_t total = n * kd;
        const unsigned grid = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
        hipLaunchKernelGGL(sym_check_kernel, dim3(grid), dim3(256), 0, s, dA, n, lda, kd, d_flag);
        BANDLU_CHECK_LAUNCH("band_is_symmetric");
    }
    return BANDLU_OK;
}

extern "C" int band_pbtrf(int64_t n, int64_t kd, double *dAB, int64_t ldab, int32_t *d_info,
                          void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 1, "band_pbtrf: n < 0");
    BANDLU_ARG(kd >= 0 && kd <= (n > 1 ? n - 1 : 0), 2, "band_pbtrf: kd out of [0, max(0, n-1)]");
    BANDLU_ARG(n == 0 || dAB != nullptr, 3, "band_pbtrf: dAB is null");
    BANDLU_ARG(ldab >= kd + 1, 4, "band_pbtrf: ldab < kd+1");
    BANDLU_ARG(d_info != nullptr, 5, "band_pbtrf: d_info is null");
    if (n > INT_MAX) {
        set_error("band_pbtrf: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return pbtrf(n, kd, dAB, ldab, ldab * n, d_info, 1, as_stream(stream));
}

extern "C" int band_pbtrf_batched(int64_t n, int64_t kd, double *dAB, int64_t ldab,
                                  int64_t strideAB, int32_t *d_info, int64_t batch, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 1, "band_pbtrf_batched: n < 0");
    BANDLU_ARG(kd >= 0 && kd <= (n > 1 ? n - 1 : 0), 2, "band_pbtrf_batched: kd out of range");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 3, "band_pbtrf_batched: dAB is null");
    BANDLU_ARG(ldab >= kd + 1, 4, "band_pbtrf_batched: ldab < kd+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 5, "band_pbtrf_batched: strideAB < ldab*n");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 6, "band_pbtrf_batched: d_info is null");
    BANDLU_ARG(batch >= 0, 7, "band_pbtrf_batched: batch < 0");
    if (n > INT_MAX || batch > INT_MAX) {
        set_error("band_pbtrf_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return pbtrf(n, kd, dAB, ldab, strideAB, d_info, batch, as_stream(stream));
}

extern "C" int band_pbtrs(int64_t n, int64_t kd, int64_t nrhs, const double *dAB, int64_t ldab,
                          double *dB, int64_t ldb, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 1, "band_pbtrs: n < 0");
    BANDLU_ARG(kd >= 0 && kd <= (n > 1 ? n - 1 : 0), 2, "band_pbtrs: kd out of range");
    BANDLU_ARG(nrhs >= 0, 3, "band_pbtrs: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 4, "band_pbtrs: dAB is null");
    BANDLU_ARG(ldab >= kd + 1, 5, "band_pbtrs: ldab < kd+1");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 6, "band_pbtrs: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 7, "band_pbtrs: ldb < max(1, n)");
    if (n > kMaxN || nrhs > INT_MAX) {
        set_error("band_pbtrs: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return pbtrs(n, kd, nrhs, dAB, ldab, ldab * n, dB, ldb, ldb * nrhs, 1, as_stream(stream));
}

extern "C" int band_pbtrs_batched(int64_t n, int64_t kd, int64_t nrhs, const double *dAB,
                                  int64_t ldab, int64_t strideAB, double *dB, int64_t ldb,
                                  int64_t strideB, int64_t batch, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 1, "band_pbtrs_batched: n < 0");
    BANDLU_ARG(kd >= 0 && kd <= (n > 1 ? n - 1 : 0), 2, "band_pbtrs_batched: kd out of range");
    BANDLU_ARG(nrhs >= 0, 3, "band_pbtrs_batched: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 4, "band_pbtrs_batched: dAB is null");
    BANDLU_ARG(ldab >= kd + 1, 5, "band_pbtrs_batched: ldab < kd+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 6, "band_pbtrs_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 7,
               "band_pbtrs_batched: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 8, "band_pbtrs_batched: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 9, "band_pbtrs_batched: strideB < ldb*nrhs");
    BANDLU_ARG(batch >= 0, 10, "band_pbtrs_batched: batch < 0");
    if (n > kMaxN || batch > INT_MAX || nrhs > INT_MAX || batch * nrhs > INT_MAX) {
        set_error("band_pbtrs_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return pbtrs(n, kd, nrhs, dAB, ldab, strideAB, dB, ldb, strideB, batch, as_stream(stream));
}
