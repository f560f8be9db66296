// Solve with the band factors (xGBTRS, no transpose): the "lu(A) \ B" that
// Listings 1 and 2 end with.
//
// One wavefront solves one right-hand side of one system.  The right-hand
// side lives in LDS when it fits (else it is updated in place in global
// memory); lane t applies the update of row j+t (forward, t = 1..kl) or row
// j-t (backward, t = 1..kl+ku).  The factor column each step needs is loaded
// D steps ahead into a register ring, so the step chain never waits on HBM.
#include <algorithm>

#include "common.hpp"

#include <utility>

namespace bandlu {
namespace {

struct RsParams {
    const double *AB;
    const int32_t *ipiv;
    double *B;
    int64_t n, kl, ku, nrhs, ldab, strideAB, strideP, ldb, strideB;
};

constexpr int64_t kLdsMaxN = 8192;  // 64 KiB of LDS per right-hand side

template <int W, int D, bool LDS>
__global__ __launch_bounds__(64) void getrs_kernel(RsParams P) {
    extern __shared__ double smem[];
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    const int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    double *Bg = P.B + b * P.strideB + k * P.ldb;
    double *x = LDS ? smem : Bg;
    const int lane = threadIdx.x;
    const int64_t n = P.n, kl = P.kl, kv = P.kl + P.ku, ldab = P.ldab;
    if (LDS) {
        for (int64_t i = lane; i < n; i += 64) x[i] = Bg[i];
        __syncthreads();
    }
    // forward: L with the row interchanges
    if (kl > 0 && n > 1) {
        auto lfetch = [&](int64_t j, int w) -> double {
            const int64_t t = 1 + lane + 64 * w;
            return (j < n - 1 && t <= min(kl, n - 1 - j)) ? AB[j * ldab + kv + t] : 0.0;
        };
        double lr[D][W];
        int ip[D];
#pragma unroll
        for (int u = 0; u < D; ++u) {
#pragma unroll
            for (int w = 0; w < W; ++w) lr[u][w] = lfetch(u, w);
            ip[u] = u < n - 1 ? ipiv[u] : 0;
        }
        for (int64_t j0 = 0; j0 < n - 1; j0 += D) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int64_t j = j0 + u;
                        if (j >= n - 1) return;
                        int64_t l = ip[u] - 1;
                        if (l < j || l >= n) l = j;  // never touch memory off the vector
                        if (lane == 0 && l != j) {
                            const double t = x[l];
                            x[l] = x[j];
                            x[j] = t;
                        }
                        __syncthreads();
                        const double bj = x[j];
                        const int64_t km = min(kl, n - 1 - j);
#pragma unroll
                        for (int w = 0; w < W; ++w) {
                            const int64_t t = 1 + lane + 64 * w;
                            if (t <= km) x[j + t] = __builtin_fma(-lr[u][w], bj, x[j + t]);
                        }
                        __syncthreads();
#pragma unroll
                        for (int w = 0; w < W; ++w) lr[u][w] = lfetch(j + D, w);
                        ip[u] = j + D < n - 1 ? ipiv[j + D] : 0;
                    }(),
                    ...);
            }(std::make_integer_sequence<int, D>{});
        }
    }
    // backward: U with kl+ku superdiagonals
    {
        auto ufetch = [&](int64_t j, int w) -> double {
            const int64_t t = lane + 64 * w;
            return (j >= 0 && t <= min(kv, j)) ? AB[j * ldab + kv - t] : 0.0;
        };
        double ur[D][W];
#pragma unroll
        for (int u = 0; u < D; ++u)
#pragma unroll
            for (int w = 0; w < W; ++w) ur[u][w] = ufetch(n - 1 - u, w);
        for (int64_t j0 = n - 1; j0 >= 0; j0 -= D) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int64_t j = j0 - u;
                        if (j < 0) return;
                        if (lane == 0) x[j] = x[j] / ur[u][0];
                        __syncthreads();
                        const double bj = x[j];
                        const int64_t tm = min(kv, j);
#pragma unroll
                        for (int w = 0; w < W; ++w) {
                            const int64_t t = lane + 64 * w;
                            if (t >= 1 && t <= tm) x[j - t] = __builtin_fma(-ur[u][w], bj, x[j - t]);
                        }
                        __syncthreads();
#pragma unroll
                        for (int w = 0; w < W; ++w) ur[u][w] = ufetch(j - D, w);
                    }(),
                    ...);
            }(std::make_integer_sequence<int, D>{});
        }
    }
    if (LDS) {
        for (int64_t i = lane; i < n; i += 64) Bg[i] = x[i];
    }
}

template <int W>
constexpr int rs_depth() { return W >= 16 ? 2 : 32 / W; }

template <int W>
int launch_w(bool lds, const RsParams &P, int64_t systems, hipStream_t s) {
    constexpr int D = rs_depth<W>();
    if (lds) {
        hipLaunchKernelGGL((getrs_kernel<W, D, true>), dim3((unsigned)systems), dim3(64),
                           size_t(P.n) * sizeof(double), s, P);
    } else {
        hipLaunchKernelGGL((getrs_kernel<W, D, false>), dim3((unsigned)systems), dim3(64), 0, s,
                           P);
    }
    BANDLU_CHECK_LAUNCH("band_getrs");
    return BANDLU_OK;
}

int launch_getrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                 int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                 double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    RsParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.B = dB;
    P.n = n;
    P.kl = kl;
    P.ku = ku;
    P.nrhs = nrhs;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    P.ldb = ldb;
    P.strideB = strideB;
    const int64_t systems = batch * nrhs;
    if (systems > INT32_MAX) {
        set_error("band_getrs: batch * nrhs too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    const int64_t lanes_needed = std::max(kl, kl + ku + 1);
    const bool lds = n <= kLdsMaxN;
    if (lanes_needed <= 64) return launch_w<1>(lds, P, systems, s);
    if (lanes_needed <= 128) return launch_w<2>(lds, P, systems, s);
    if (lanes_needed <= 256) return launch_w<4>(lds, P, systems, s);
    if (lanes_needed <= 512) return launch_w<8>(lds, P, systems, s);
    if (lanes_needed <= 1024) return launch_w<16>(lds, P, systems, s);
    set_error("band_getrs: kl + ku + 1 > 1024 is not supported");
    return BANDLU_ERR_UNSUPPORTED;
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int band_getrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                          int64_t ldab, const int32_t *d_ipiv, double *dB, int64_t ldb,
                          void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_getrs: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || d_ipiv != nullptr, 7, "band_getrs: d_ipiv is null");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 8, "band_getrs: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 9, "band_getrs: ldb < max(1, n)");
    if (n > kMaxN) {
        set_error("band_getrs: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrs(n, kl, ku, nrhs, dAB, ldab, ldab * n, d_ipiv, n, dB, ldb, ldb * nrhs, 1,
                        as_stream(stream));
}

extern "C" int band_getrs_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs,
                                  const double *dAB, int64_t ldab, int64_t strideAB,
                                  const int32_t *d_ipiv, int64_t strideP, double *dB,
                                  int64_t ldb, int64_t strideB, int64_t batch, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs_batched: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs_batched: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_getrs_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_getrs_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 8, "band_getrs_batched: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 9, "band_getrs_batched: strideP < n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 10,
               "band_getrs_batched: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 11, "band_getrs_batched: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 12, "band_getrs_batched: strideB < ldb*nrhs");
    BANDLU_ARG(batch >= 0, 13, "band_getrs_batched: batch < 0");
    if (n > kMaxN) {
        set_error("band_getrs_batched: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_getrs(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb, strideB,
                        batch, as_stream(stream));
}
