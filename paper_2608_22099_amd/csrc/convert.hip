// Step 2 of the structure-aware strategy (Sec. II-A, cost C(N); Listing 2's
// conversion of the dense matrix to a band matrix): pack a dense column-major
// matrix into the xGBTRF band layout.
//
// Band column j (rows 0..2kl+ku) is contiguous in AB and its in-band source
// rows j-ku..j+kl are contiguous in column j of A, so the copy is a gather of
// one contiguous segment per column with no transpose: a lane maps to one band
// slot, reads its source element (or produces +0.0 for a fill or corner slot)
// and writes it, and consecutive lanes write consecutive band slots.  When a
// band column is at most 32 slots tall several columns share one wavefront so
// that stores stay wide.  Each wavefront owns a contiguous run of columns of
// the batch; values move as 64-bit integers, so every bit pattern survives.
#include <algorithm>

#include "common.hpp"

namespace bandlu {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

struct ConvParams {
    const unsigned long long *A;
    unsigned long long *AB;
    int64_t n, lda, strideA, kl, ku, ldab, strideAB;
    int64_t total_cols, cols_per_wave;
    int rows;          // 2kl + ku + 1
    int per;           // band columns per wave step (rows <= 32), else 1
    int64_t per_div_n, per_mod_n;
};

__device__ inline unsigned long long conv_value(const ConvParams &P, int64_t b, int64_t j, int r) {
    const int64_t i = j - P.kl - P.ku + r;
    if (r >= P.kl && i >= 0 && i < P.n) return P.A[b * P.strideA + j * P.lda + i];
    return 0ull;
}

// rows <= 32: lane -> (column offset lane / rows, band row lane % rows)
__global__ __launch_bounds__(kThreads) void conv_packed(ConvParams P) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t(blockIdx.x) * kThreads + threadIdx.x) >> 6;
    const int64_t g0 = wave * P.cols_per_wave;
    const int64_t g1 = min(g0 + P.cols_per_wave, P.total_cols);
    if (g0 >= g1) return;
    const int qc = lane / P.rows;
    const int r = lane - qc * P.rows;
    if (qc >= P.per) return;
    int64_t g = g0 + qc;
    int64_t b = g / P.n;
    int64_t j = g - b * P.n;
    while (g < g1) {
        unsigned long long v[kUnroll];
        int64_t bb[kUnroll], jj[kUnroll];
        bool ok[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            ok[u] = g < g1;
            bb[u] = b;
            jj[u] = j;
            v[u] = ok[u] ? conv_value(P, b, j, r) : 0ull;
            g += P.per;
            b += P.per_div_n;
            j += P.per_mod_n;
            if (j >= P.n) { j -= P.n; ++b; }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (ok[u]) P.AB[bb[u] * P.strideAB + jj[u] * P.ldab + r] = v[u];
    }
}

// rows > 32: one band column per wave step, lanes stride over its rows
__global__ __launch_bounds__(kThreads) void conv_tall(ConvParams P) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t(blockIdx.x) * kThreads + threadIdx.x) >> 6;
    const int64_t g0 = wave * P.cols_per_wave;
    const int64_t g1 = min(g0 + P.cols_per_wave, P.total_cols);
    if (g0 >= g1) return;
    int64_t b = g0 / P.n;
    int64_t j = g0 - b * P.n;
    for (int64_t g = g0; g < g1; ++g) {
        unsigned long long *dst = P.AB + b * P.strideAB + j * P.ldab;
        for (int r0 = 0; r0 < P.rows; r0 += 64 * kUnroll) {
            unsigned long long v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                int r = r0 + u * 64 + lane;
                v[u] = r < P.rows ? conv_value(P, b, j, r) : 0ull;
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                int r = r0 + u * 64 + lane;
                if (r < P.rows) dst[r] = v[u];
            }
        }
        if (++j == P.n) { j = 0; ++b; }
    }
}

int launch_convert(const double *dA, int64_t n, int64_t lda, int64_t strideA, int64_t kl,
                   int64_t ku, double *dAB, int64_t ldab, int64_t strideAB, int64_t batch,
                   hipStream_t s) {
    if (n == 0 || batch == 0) return BANDLU_OK;
    ConvParams P;
    P.A = reinterpret_cast<const unsigned long long *>(dA);
    P.AB = reinterpret_cast<unsigned long long *>(dAB);
    P.n = n;
    P.lda = lda;
    P.strideA = strideA;
    P.kl = kl;
    P.ku = ku;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.total_cols = n * batch;
    const int64_t rows = 2 * kl + ku + 1;
    P.rows = (int)rows;
    P.per = rows <= 32 ? int(64 / rows) : 1;
    P.per_div_n = P.per / n;
    P.per_mod_n = P.per % n;
    // wave steps of `per` columns; aim for 8 waves per SIMD
    const int64_t max_waves = int64_t(device_cu_count()) * 32;
    const int64_t steps = (P.total_cols + P.per - 1) / P.per;
    const int64_t waves = std::min(steps, max_waves);
    int64_t steps_per_wave = (steps + waves - 1) / waves;
    P.cols_per_wave = steps_per_wave * P.per;
    const int64_t used_waves = (P.total_cols + P.cols_per_wave - 1) / P.cols_per_wave;
    const int64_t blocks = (used_waves + (kThreads / 64) - 1) / (kThreads / 64);
    if (rows <= 32)
        hipLaunchKernelGGL(conv_packed, dim3((unsigned)blocks), dim3(kThreads), 0, s, P);
    else
        hipLaunchKernelGGL(conv_tall, dim3((unsigned)blocks), dim3(kThreads), 0, s, P);
    BANDLU_CHECK_LAUNCH("dense_to_band");
    return BANDLU_OK;
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int dense_to_band(const double *dA, int64_t n, int64_t lda, int64_t kl, int64_t ku,
                             double *dAB, int64_t ldab, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 2, "dense_to_band: n = %lld < 0", (long long)n);
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "dense_to_band: lda < max(1, n)");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 4, "dense_to_band: kl out of [0, max(0, n-1)]");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 5, "dense_to_band: ku out of [0, max(0, n-1)]");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 7, "dense_to_band: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || dA != nullptr, 1, "dense_to_band: dA is null");
    BANDLU_ARG(n == 0 || dAB != nullptr, 6, "dense_to_band: dAB is null");
    if (n > kMaxN) {
        set_error("dense_to_band: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_convert(dA, n, lda, lda * n, kl, ku, dAB, ldab, ldab * n, 1,
                          as_stream(stream));
}

extern "C" int dense_to_band_batched(const double *dA, int64_t n, int64_t lda, int64_t strideA,
                                     int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                                     int64_t strideAB, int64_t batch, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 2, "dense_to_band_batched: n < 0");
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "dense_to_band_batched: lda < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideA >= lda * n, 4, "dense_to_band_batched: strideA < lda*n");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 5, "dense_to_band_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 6, "dense_to_band_batched: ku out of range");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 8, "dense_to_band_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 9, "dense_to_band_batched: strideAB < ldab*n");
    BANDLU_ARG(batch >= 0, 10, "dense_to_band_batched: batch < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dA != nullptr, 1, "dense_to_band_batched: dA is null");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 7, "dense_to_band_batched: dAB is null");
    if (n > kMaxN || (n > 0 && batch > INT64_MAX / n)) {
        set_error("dense_to_band_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_convert(dA, n, lda, strideA, kl, ku, dAB, ldab, strideAB, batch,
                          as_stream(stream));
}
