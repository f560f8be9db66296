// Solve with the band factors (xGBTRS, no transpose): the "lu(A) \ B" that
// Listings 1 and 2 end with.
//
// One wavefront solves one right-hand side of one system.  The right-hand
// side lives in LDS when it fits (else it is updated in place in global
// memory); lane t applies the update of row j+t (forward, t = 1..kl) or row
// j-t (backward, t = 1..kl+ku).  The factor column each step needs is loaded
// D steps ahead into a register ring, so the step chain never waits on HBM.
#include <algorithm>

#include "bufio.hpp"
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

// Register-window solve for narrow bands (kl <= 63, kl + ku < 64 * CPL).
// Forward: row r of the right-hand side lives in lane r mod 64; at step j lane
// j mod 64 holds b[j], the swap with row ipiv[j]-1 is an exchange between two
// lanes, and lanes holding rows j+1..j+kl apply one fma each.  Backward: row r
// lives in lane r mod 64, register sub-slot (r / 64) mod CPL; at step j the
// lane holding b[j] divides by U(j,j) and lanes holding rows j-kl-ku..j-1 apply
// one fma each.  Multipliers, U entries, pivot indices and rows entering the
// window are loaded D steps ahead into register rings whose index is a
// compile-time constant (the step loop is unrolled by 64 * CPL).  Every step is
// straight-line code: memory goes through range-checked buffer operations and
// lane predicates are selects, so the prefetch ring stays in flight.
template <int CPL>
__global__ __launch_bounds__(64) void getrs_win_kernel(RsParams P) {
    constexpr int D = 16;
    constexpr int M = 64 * CPL;
    const int L = threadIdx.x;
    const int64_t sys = blockIdx.x;
    const int64_t bidx = sys / P.nrhs, k = sys - bidx * P.nrhs;
    const int n = int(P.n), kl = int(P.kl), kv = int(P.kl + P.ku), ldab = int(P.ldab);
    const Buf ab = make_buf(P.AB + bidx * P.strideAB, uint32_t(int64_t(ldab) * n * 8));
    const Buf pb = make_buf(P.ipiv + bidx * P.strideP, uint32_t(int64_t(n) * 4));
    const Buf xb = make_buf(P.B + bidx * P.strideB + k * P.ldb, uint32_t(int64_t(n) * 8));
    auto rowoff = [](int r) -> uint32_t { return uint32_t(r) * 8u; };  // r < 0 or r >= n: outside

    // ------------------------------------------------------------ forward --
    if (kl > 0 && n > 1) {
        double bv = buf_ld(xb, L <= kl ? rowoff(L) : kOutside);
        auto loff = [&](int j) -> uint32_t {  // multiplier for this lane's row at step j
            const int t = (L - j) & 63;
            const bool ok = j < n - 1 && t >= 1 && t <= min(kl, n - 1 - j);
            return ok ? uint32_t(j * ldab + kv + t) * 8u : kOutside;
        };
        double lr[D], rr[D];
#pragma unroll
        for (int d = 0; d < D; ++d) {
            lr[d] = buf_ld(ab, loff(d));
            rr[d] = buf_ld(xb, rowoff(kl + 1 + d));
        }
        int ipv = buf_ld_i32(pb, uint32_t(L) * 4u);
        int ipv_next = buf_ld_i32(pb, uint32_t(L + 64) * 4u);
        for (int j0 = 0; j0 < n - 1; j0 += 64) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int j = j0 + u;
                        const bool live = j < n - 1;
                        int l = __builtin_amdgcn_readlane(ipv, u) - 1;
                        l = (live && l > j && l <= j + kl && l < n) ? l : j;
                        if (l != j) {
                            const int ls = l & 63;
                            const double vj = readlane_d(bv, u);
                            const double vl = readlane_d(bv, ls);
                            bv = L == u ? vl : (L == ls ? vj : bv);
                        }
                        const double bj = readlane_d(bv, u);
                        const int t = (L - u) & 63;
                        const bool m = t >= 1 && t <= min(kl, n - 1 - j);
                        const double nb = __builtin_fma(-lr[u % D], bj, bv);
                        bv = m ? nb : bv;
                        buf_st(xb, (L == u && live) ? rowoff(j) : kOutside, bv);  // row j is final
                        const int renter = j + kl + 1;
                        bv = (live && L == (renter & 63) && renter < n) ? rr[u % D] : bv;
                        lr[u % D] = buf_ld(ab, loff(j + D));
                        rr[u % D] = buf_ld(xb, rowoff(renter + D));
                        if constexpr (u == 63) {
                            ipv = ipv_next;
                            ipv_next = buf_ld_i32(pb, uint32_t(j0 + 128 + L) * 4u);
                        }
                    }(),
                    ...);
            }(std::make_integer_sequence<int, 64>{});
        }
        buf_st(xb, L == ((n - 1) & 63) ? rowoff(n - 1) : kOutside, bv);
        __threadfence();
    }
    // ----------------------------------------------------------- backward --
    {
        auto rowof = [&](int s, int j) -> int { return j - ((j - (L + 64 * s)) & (M - 1)); };
        double bv[CPL];
#pragma unroll
        for (int s = 0; s < CPL; ++s) {
            const int r = rowof(s, n - 1);
            bv[s] = buf_ld(xb, r >= n - 1 - kv ? rowoff(r) : kOutside);
        }
        auto uoff = [&](int s, int j) -> uint32_t {  // U(row, j) for this lane's row at step j
            const int t = j - rowof(s, j);
            const bool ok = j >= 0 && t >= 1 && t <= min(kv, j);
            return ok ? uint32_t(j * ldab + kv - t) * 8u : kOutside;
        };
        auto doff = [&](int j) -> uint32_t { return j >= 0 ? uint32_t(j * ldab + kv) * 8u : kOutside; };
        double ur[CPL][D], dr[D], rr[D];
#pragma unroll
        for (int d = 0; d < D; ++d) {
#pragma unroll
            for (int s = 0; s < CPL; ++s) ur[s][d] = buf_ld(ab, uoff(s, n - 1 - d));
            dr[d] = buf_ld(ab, doff(n - 1 - d));
            rr[d] = buf_ld(xb, rowoff(n - 2 - kv - d));
        }
        // steps are counted from the end so that register indices are constants
        for (int m0 = 0; m0 < n; m0 += M) {
            [&]<int... Us>(std::integer_sequence<int, Us...>) {
                (
                    [&] {
                        constexpr int u = Us;
                        const int j = n - 1 - (m0 + u);
                        const bool live = j >= 0;
                        const int lj = j & 63;
                        const int sj = (j >> 6) & (CPL - 1);
                        double zs = bv[0];
#pragma unroll
                        for (int s = 1; s < CPL; ++s) zs = sj == s ? bv[s] : zs;
                        const double z = zs / dr[u % D];
                        const double xj = readlane_d(z, lj);
                        buf_st(xb, (live && L == lj) ? rowoff(j) : kOutside, xj);
#pragma unroll
                        for (int s = 0; s < CPL; ++s) {
                            const int t = j - rowof(s, j);
                            const bool m = t >= 1 && t <= min(kv, j);
                            const double nb = __builtin_fma(-ur[s][u % D], xj, bv[s]);
                            bv[s] = m ? nb : bv[s];
                        }
                        const int renter = j - 1 - kv;
                        const bool ent = live && renter >= 0 && L == (renter & 63);
                        const int se = (renter >> 6) & (CPL - 1);
#pragma unroll
                        for (int s = 0; s < CPL; ++s) bv[s] = (ent && se == s) ? rr[u % D] : bv[s];
#pragma unroll
                        for (int s = 0; s < CPL; ++s) ur[s][u % D] = buf_ld(ab, uoff(s, j - D));
                        dr[u % D] = buf_ld(ab, doff(j - D));
                        rr[u % D] = buf_ld(xb, rowoff(renter - D));
                    }(),
                    ...);
            }(std::make_integer_sequence<int, M>{});
        }
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
    const bool buf_ok = ldab * n * 8 <= kMaxBufferBytes && n * 8 <= kMaxBufferBytes;
    if (buf_ok && kl <= 63 && kl + ku < 64) {
        hipLaunchKernelGGL(getrs_win_kernel<1>, dim3((unsigned)systems), dim3(64), 0, s, P);
        BANDLU_CHECK_LAUNCH("band_getrs (window)");
        return BANDLU_OK;
    }
    if (buf_ok && kl <= 63 && kl + ku < 128) {
        hipLaunchKernelGGL(getrs_win_kernel<2>, dim3((unsigned)systems), dim3(64), 0, s, P);
        BANDLU_CHECK_LAUNCH("band_getrs (window)");
        return BANDLU_OK;
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
