// Substitutions built on the chain of column steps (getrs_ring.hpp):
//
//  * Listing 1's triangular and diagonal branches (Sec. I-C): a band whose
//    detected ku is 0 (lower triangular), kl is 0 (upper) or both (diagonal)
//    is solved straight from the converted band, with no factorisation:
//    lower = the dividing forward chain over the band's columns, upper = the
//    backward chain, diagonal = one division per entry.
//  * The transposed solve A^T x = b with the band LU factors (the general
//    "A \ B" of Listing 1 on A^T; xGBTRS with trans = 'T'):
//      U^T pass: the dividing forward chain over the rows of U (entry e of
//        step j is U(j, j+e), ldab-1 apart in the band): each x_i updates the
//        later positions in increasing i, the order of the dot products of the
//        definition, so the result is bitwise that of the reference loops;
//      L^T pass: backward, a dot product of column j's multipliers with the
//        later positions, then the interchange of row j.  The interchange
//        after each dot product rules out the update form, so one wavefront
//        per right-hand side keeps a sliding window of the vector in LDS and
//        sums each dot product in the order of the definition.
//  * The chains for bands beyond the ring's registers (K > 1023): one
//    workgroup per right-hand side, two barriers per step.
#include <algorithm>
#include <climits>

#include "getrs_ring.hpp"

namespace bandlu {

int launch_chain(int mode, const RingParams &P, int64_t batch, hipStream_t s);
int launch_getrf_wide(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                      int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                      int64_t batch, hipStream_t s, void *scratch, size_t scratch_bytes,
                      double *dB, int64_t ldb, int64_t strideB, int64_t nrhs);
bool getrf_wide_fused_fits(int64_t n, int64_t kl, int64_t ku, int64_t nrhs);
int launch_getrf_lean_fwd(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int32_t *d_ipiv, double *dB, int32_t *d_info, hipStream_t s);

namespace {

constexpr int kAnyThreads = 256;
constexpr int64_t kChainLdsMaxN = 8192;  // vector in LDS up to 64 KiB

// One pass for any K: position q is row q (forward) or n-1-q (backward).
template <int MODE, bool LDS>
__global__ __launch_bounds__(kAnyThreads) void chain_any_kernel(RingParams P) {
    extern __shared__ double smem[];
    constexpr bool BWD = MODE == kRingBwd;
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    double *Bg = P.B + b * P.strideB + k * P.ldb;
    double *x = LDS ? smem : Bg;
    const int tid = threadIdx.x;
    const int64_t n = P.n, K = P.K, ldab = P.ldab;
    if (LDS) {
        for (int64_t i = tid; i < n; i += kAnyThreads) x[i] = Bg[i];
    }
    __syncthreads();
    const int32_t *ipiv = MODE == kRingFwdLU ? P.ipiv + b * P.strideP : nullptr;
    for (int64_t j = 0; j < P.nsteps; ++j) {
        const int64_t col = BWD ? n - 1 - j : j;
        const int64_t rj = BWD ? n - 1 - j : j;
        const double *cb = AB + P.cb0 + col * ldab;
        if (tid == 0) {
            if constexpr (MODE == kRingFwdLU) {
                // the row interchange of step j (unit diagonal: no division)
                const int64_t l = ipiv[j] - 1;
                if (l != j && l > j && l < n) {
                    const double t0 = x[l];
                    x[l] = x[j];
                    x[j] = t0;
                }
            } else {
                x[rj] = x[rj] / cb[(BWD ? K : 0) * P.es];
            }
        }
        __syncthreads();
        const double xj = x[rj];
        const int64_t dmax = std::min(K, n - 1 - j);
        for (int64_t d = 1 + tid; d <= dmax; d += kAnyThreads) {
            const int64_t e = BWD ? K - d : d;
            const int64_t r = BWD ? rj - d : rj + d;
            x[r] = __builtin_fma(-cb[e * P.es], xj, x[r]);
        }
        __syncthreads();
    }
    if (LDS) {
        for (int64_t i = tid; i < n; i += kAnyThreads) Bg[i] = x[i];
    }
}

// L^T pass of the transposed solve.  One wavefront per right-hand side; the
// positions between the lowest one loaded and the lowest one stored live in
// an LDS ring of R doubles (R a power of two >= kl + 192).  Step j (n-2 down
// to 0) reads positions j..j+km; afterwards positions >= j + kl are final.
struct LtParams {
    const double *AB;
    const int32_t *ipiv;
    double *B;
    int64_t ldab, strideAB, strideP, ldb, strideB;
    int n, kl, kv, nrhs, R;
};

__global__ __launch_bounds__(64) void lt_swap_kernel(LtParams P) {
    extern __shared__ double ring[];
    const int lane = threadIdx.x;
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    const int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    double *x = P.B + b * P.strideB + k * P.ldb;
    const int n = P.n, kl = P.kl, mask = P.R - 1;
    const int64_t ldab = P.ldab;
    int low = std::max(0, n - 64);  // lowest position loaded
    int hi = n;                     // positions >= hi are stored back
    if (low + lane < n) ring[(low + lane) & mask] = x[low + lane];
    int ipv = 0, ipv_base = -1;
    // multipliers of the next step's column, the first kPre*64 (prefetched a
    // step ahead, so that no step waits for a load)
    constexpr int kPre = 4;
    auto lcol = [&](int j, int ch) -> double {
        const int km = std::min(kl, n - 1 - j);
        const int t = 1 + 64 * ch + lane;
        return (j >= 0 && t <= km) ? AB[P.kv + t + int64_t(j) * ldab] : 0.0;
    };
    double lnext[kPre];
#pragma unroll
    for (int ch = 0; ch < kPre; ++ch) lnext[ch] = lcol(n - 2, ch);
    __syncthreads();
    for (int j = n - 2; j >= 0; --j) {
        if (j < low) {
            const int nl = std::max(0, low - 64);
            if (nl + lane < low) ring[(nl + lane) & mask] = x[nl + lane];
            low = nl;
            __syncthreads();
        }
        if (j < ipv_base || ipv_base < 0) {
            ipv_base = std::max(0, j - 63);
            ipv = ipv_base + lane <= j ? ipiv[ipv_base + lane] : 0;
        }
        const int km = std::min(kl, n - 1 - j);
        double lcur[kPre];
#pragma unroll
        for (int ch = 0; ch < kPre; ++ch) {
            lcur[ch] = lnext[ch];
            lnext[ch] = lcol(j - 1, ch);
        }
        double acc = ring[j & mask];
        for (int t0 = 1, ch = 0; t0 <= km; t0 += 64, ++ch) {
            double lv = 0.0;
#pragma unroll
            for (int c2 = 0; c2 < kPre; ++c2)
                if (ch == c2) lv = lcur[c2];
            if (ch >= kPre) lv = lcol(j, ch);
            const double v = t0 + lane <= km ? ring[(j + t0 + lane) & mask] : 0.0;
            const int cnt = std::min(64, km - t0 + 1);
            // (the chain of fused multiply-adds in the order of the definition;
            // unrolled by eight so that the lane reads of the next terms issue
            // while an fma waits)
            for (int u0 = 0; u0 < cnt; u0 += 8) {
#pragma unroll
                for (int u1 = 0; u1 < 8; ++u1) {
                    const int u = u0 + u1;
                    if (u < cnt) acc = __builtin_fma(-readlane_d(lv, u), readlane_d(v, u), acc);
                }
            }
        }
        const int p = __builtin_amdgcn_readlane(ipv, j - ipv_base) - 1;
        if (lane == 0) {
            if (p != j && p > j && p < n) {
                const double vp = ring[p & mask];
                ring[p & mask] = acc;
                ring[j & mask] = vp;
            } else {
                ring[j & mask] = acc;
            }
        }
        __syncthreads();
        // positions >= j + kl are final: store a block of 64 once it is complete
        if (hi - 64 >= j + kl && hi - 64 >= 0) {
            x[hi - 64 + lane] = ring[(hi - 64 + lane) & mask];
            hi -= 64;
        }
    }
    __syncthreads();
    for (int q = lane; q < hi; q += 64) x[q] = ring[q & mask];
}

// The same pass for kl <= 1024 with both operands of every term in LDS: each
// step's multipliers are staged next to the window (all lanes write their
// prefetched part), the window keeps two copies of every position (at q mod R
// and R + q mod R, so positions j+1 .. j+km are consecutive), and the chain of
// fused multiply-adds reads two terms per LDS load, the same in every lane
// (no lane reads, no copies to vector registers).  The sums are those of the
// definition in its order, so the result is lt_swap_kernel's.
constexpr int kLtDotMaxKl = 1024;

// keeps the compiler from sinking the next block's LDS loads below this point
__device__ __forceinline__ void lt_fence() { asm volatile("" ::: "memory"); }

__global__ __launch_bounds__(64) void lt_dot_kernel(LtParams P) {
    extern __shared__ double lds_lt[];
    const int lane = threadIdx.x;
    const int64_t sys = blockIdx.x;
    const int64_t b = sys / P.nrhs, k = sys - b * P.nrhs;
    const double *__restrict__ AB = P.AB + b * P.strideAB;
    const int32_t *__restrict__ ipiv = P.ipiv + b * P.strideP;
    double *x = P.B + b * P.strideB + k * P.ldb;
    const int n = P.n, kl = P.kl, R = P.R, mask = R - 1;
    double *const ring = lds_lt;           // 2R doubles
    double *const lbuf = lds_lt + 2 * R;   // the step's multipliers, kl rounded up to 64
    const int64_t ldab = P.ldab;
    auto put = [&](int q, double v) {
        ring[q & mask] = v;
        ring[(q & mask) + R] = v;
    };
    int low = std::max(0, n - 64);  // lowest position loaded
    int hi = n;                     // positions >= hi are stored back
    if (low + lane < n) put(low + lane, x[low + lane]);
    int ipv = 0, ipv_base = -1;
    constexpr int kPre = 4;  // chunks of 64 multipliers prefetched a step ahead
    const int nch = (kl + 63) / 64;
    auto lcol = [&](int j, int ch) -> double {
        const int km = std::min(kl, n - 1 - j);
        const int t = 1 + 64 * ch + lane;
        return (j >= 0 && t <= km) ? AB[P.kv + t + int64_t(j) * ldab] : 0.0;
    };
    double lnext[kPre];
#pragma unroll
    for (int ch = 0; ch < kPre; ++ch) lnext[ch] = lcol(n - 2, ch);
    __syncthreads();
    for (int j = n - 2; j >= 0; --j) {
        if (j < low) {
            const int nl = std::max(0, low - 64);
            if (nl + lane < low) put(nl + lane, x[nl + lane]);
            low = nl;
        }
        if (j < ipv_base || ipv_base < 0) {
            ipv_base = std::max(0, j - 63);
            ipv = ipv_base + lane <= j ? ipiv[ipv_base + lane] : 0;
        }
        const int km = std::min(kl, n - 1 - j);
        // stage column j's multipliers (term t = 1 + u at lbuf[u]) and take
        // column j-1's into the prefetch registers
#pragma unroll
        for (int ch = 0; ch < kPre; ++ch) {
            if (ch < nch) lbuf[64 * ch + lane] = lnext[ch];
            lnext[ch] = lcol(j - 1, ch);
        }
        for (int ch = kPre; ch < nch; ++ch) lbuf[64 * ch + lane] = lcol(j, ch);
        __syncthreads();
        const double *const w = ring + ((j + 1) & mask);
        double acc = ring[j & mask];
        const int nfull = km >> 6;
        for (int ch = 0; ch < nfull; ++ch) {
            const double *const lw = lbuf + 64 * ch;
            const double *const xw = w + 64 * ch;
            // blocks of 16 terms, the loads of the next block issued before
            // the fused multiply-adds of this one (the LDS latency is then
            // under the chain)
            double la[2][16], xa[2][16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                la[0][u] = lw[u];
                xa[0][u] = xw[u];
            }
#pragma unroll
            for (int blk = 0; blk < 4; ++blk) {
                if (blk + 1 < 4) {
#pragma unroll
                    for (int u = 0; u < 16; ++u) {
                        la[(blk + 1) & 1][u] = lw[16 * (blk + 1) + u];
                        xa[(blk + 1) & 1][u] = xw[16 * (blk + 1) + u];
                    }
                }
                lt_fence();
#pragma unroll
                for (int u = 0; u < 16; ++u) acc = __builtin_fma(-la[blk & 1][u], xa[blk & 1][u], acc);
            }
        }
        for (int u = 64 * nfull; u < km; ++u) acc = __builtin_fma(-lbuf[u], w[u], acc);
        const int p = __builtin_amdgcn_readlane(ipv, j - ipv_base) - 1;
        if (lane == 0) {
            if (p != j && p > j && p < n) {
                const double vp = ring[p & mask];
                put(p, acc);
                put(j, vp);
            } else {
                put(j, acc);
            }
        }
        __syncthreads();
        // positions >= j + kl are final: store a block of 64 once it is complete
        if (hi - 64 >= j + kl && hi - 64 >= 0) {
            x[hi - 64 + lane] = ring[(hi - 64 + lane) & mask];
            hi -= 64;
        }
    }
    __syncthreads();
    for (int q = lane; q < hi; q += 64) x[q] = ring[q & mask];
}

__global__ void diag_div_kernel(const double *AB, int64_t ldab, int64_t strideAB, double *B,
                                int64_t ldb, int64_t strideB, int64_t n, int64_t nrhs,
                                int64_t total) {
    for (int64_t g = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; g < total;
         g += int64_t(gridDim.x) * blockDim.x) {
        const int64_t i = g % n, sys = g / n;
        const int64_t b = sys / nrhs, k = sys - b * nrhs;
        double *x = B + b * strideB + k * ldb;
        x[i] = x[i] / AB[b * strideAB + i * ldab];
    }
}

// info[b] = 1 + the first j with A(j,j) == 0 (diagonal at row kv), else 0
__global__ __launch_bounds__(256) void zero_diag_kernel(const double *AB, int64_t ldab,
                                                        int64_t strideAB, int64_t kv, int64_t n,
                                                        int32_t *info) {
    const int64_t b = blockIdx.x;
    const double *a = AB + b * strideAB + kv;
    int first = INT_MAX;
    for (int64_t j = threadIdx.x; j < n; j += 256)
        if (a[j * ldab] == 0.0) {
            first = int(j);
            break;
        }
    __shared__ int s[4];
    for (int off = 32; off >= 1; off >>= 1) first = min(first, __shfl_xor(first, off));
    if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = first;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int m = min(min(s[0], s[1]), min(s[2], s[3]));
        info[b] = m == INT_MAX ? 0 : m + 1;
    }
}

bool ring_fits_band(int64_t n, int64_t ldab, int64_t K) {
    return K >> 6 <= kMaxQ && ldab * n * 8 <= kMaxBufferBytes && n * 8 <= kMaxBufferBytes &&
           n <= INT_MAX;
}

}  // namespace

// One pass of a chain over `batch` * P.nrhs vectors: the ring for K <= 1023,
// else the any-band kernel.
int launch_chain(int mode, const RingParams &P, int64_t batch, hipStream_t s) {
    const int64_t systems = batch * P.nrhs;
    if (systems == 0 || P.nsteps <= 0) return BANDLU_OK;
    if (ring_fits_band(P.n, P.ldab, P.K)) {
        ring_pass(mode, P.K)(P, systems, s);
        BANDLU_CHECK_LAUNCH("band chain (ring)");
        return BANDLU_OK;
    }
    const bool lds = P.n <= kChainLdsMaxN;
    const size_t shm = lds ? size_t(P.n) * sizeof(double) : 0;
    if (mode == kRingBwd) {
        if (lds)
            hipLaunchKernelGGL((chain_any_kernel<kRingBwd, true>), dim3((unsigned)systems),
                               dim3(kAnyThreads), shm, s, P);
        else
            hipLaunchKernelGGL((chain_any_kernel<kRingBwd, false>), dim3((unsigned)systems),
                               dim3(kAnyThreads), 0, s, P);
    } else if (mode == kRingFwdDiv) {
        if (lds)
            hipLaunchKernelGGL((chain_any_kernel<kRingFwdDiv, true>), dim3((unsigned)systems),
                               dim3(kAnyThreads), shm, s, P);
        else
            hipLaunchKernelGGL((chain_any_kernel<kRingFwdDiv, false>), dim3((unsigned)systems),
                               dim3(kAnyThreads), 0, s, P);
    } else {
        if (lds)
            hipLaunchKernelGGL((chain_any_kernel<kRingFwdLU, true>), dim3((unsigned)systems),
                               dim3(kAnyThreads), shm, s, P);
        else
            hipLaunchKernelGGL((chain_any_kernel<kRingFwdLU, false>), dim3((unsigned)systems),
                               dim3(kAnyThreads), 0, s, P);
    }
    BANDLU_CHECK_LAUNCH("band chain (any band)");
    return BANDLU_OK;
}

namespace {

RingParams chain_params(const double *dAB, int64_t ldab, int64_t strideAB, double *dB,
                        int64_t ldb, int64_t strideB, int64_t n, int64_t nrhs) {
    RingParams P{};
    P.AB = dAB;
    P.ipiv = nullptr;
    P.B = dB;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = 0;
    P.ldb = ldb;
    P.strideB = strideB;
    P.n = (int)n;
    P.kl = 0;
    P.nrhs = (int)nrhs;
    return P;
}

int trsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB, int64_t ldab,
         int64_t strideAB, double *dB, int64_t ldb, int64_t strideB, int32_t *d_info,
         int64_t batch, hipStream_t s) {
    if (batch == 0) return BANDLU_OK;
    const int64_t kv = kl + ku;
    hipLaunchKernelGGL(zero_diag_kernel, dim3((unsigned)batch), dim3(256), 0, s, dAB, ldab,
                       strideAB, kv, n, d_info);
    BANDLU_CHECK_LAUNCH("band_trsv (info)");
    if (n == 0 || nrhs == 0) return BANDLU_OK;
    if (kl == 0 && ku == 0) {
        const int64_t total = n * nrhs * batch;
        const unsigned grid = (unsigned)std::min<int64_t>((total + 255) / 256, 8192);
        hipLaunchKernelGGL(diag_div_kernel, dim3(grid), dim3(256), 0, s, dAB, ldab, strideAB, dB,
                           ldb, strideB, n, nrhs, total);
        BANDLU_CHECK_LAUNCH("band_trsv (diagonal)");
        return BANDLU_OK;
    }
    RingParams P = chain_params(dAB, ldab, strideAB, dB, ldb, strideB, n, nrhs);
    P.nsteps = (int)n;
    if (ku == 0) {
        // lower: column j from its diagonal (row kv = kl) down
        P.cb0 = kv;
        P.es = 1;
        P.K = (int)kl;
        return launch_chain(kRingFwdDiv, P, batch, s);
    }
    // upper: column n-1-j from row 0 (A(col-ku+e, col))
    P.cb0 = 0;
    P.es = 1;
    P.K = (int)ku;
    return launch_chain(kRingBwd, P, batch, s);
}

int getrs_t(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB, int64_t ldab,
            int64_t strideAB, const int32_t *d_ipiv, int64_t strideP, double *dB, int64_t ldb,
            int64_t strideB, int64_t batch, hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    const int64_t kv = kl + ku;
    // U^T: step j reads row j of U, U(j, j+e) at kv + j*ldab + e*(ldab-1)
    RingParams P = chain_params(dAB, ldab, strideAB, dB, ldb, strideB, n, nrhs);
    P.nsteps = (int)n;
    P.cb0 = kv;
    P.es = ldab - 1;
    P.K = (int)kv;
    if (int rc = launch_chain(kRingFwdDiv, P, batch, s); rc != BANDLU_OK) return rc;
    if (kl == 0 || n < 2) return BANDLU_OK;
    LtParams T;
    T.AB = dAB;
    T.ipiv = d_ipiv;
    T.B = dB;
    T.ldab = ldab;
    T.strideAB = strideAB;
    T.strideP = strideP;
    T.ldb = ldb;
    T.strideB = strideB;
    T.n = (int)n;
    T.kl = (int)kl;
    T.kv = (int)kv;
    T.nrhs = (int)nrhs;
    int R = 256;
    while (R < kl + 192) R <<= 1;
    if (size_t(R) * sizeof(double) > 64 * 1024) {
        set_error("band_getrs_t: kl = %lld is beyond the %d the transposed solve's window holds",
                  (long long)kl, 64 * 1024 / 8 - 192);
        return BANDLU_ERR_UNSUPPORTED;
    }
    T.R = R;
    if (kl <= kLtDotMaxKl) {
        // two copies of the window and the step's multipliers (at most 40 KiB)
        const size_t lds = (size_t(2) * R + size_t((kl + 63) / 64) * 64) * sizeof(double);
        hipLaunchKernelGGL(lt_dot_kernel, dim3((unsigned)(batch * nrhs)), dim3(64), lds, s, T);
    } else {
        hipLaunchKernelGGL(lt_swap_kernel, dim3((unsigned)(batch * nrhs)), dim3(64),
                           size_t(R) * sizeof(double), s, T);
    }
    BANDLU_CHECK_LAUNCH("band_getrs_t (L^T pass)");
    return BANDLU_OK;
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int band_trsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                         int64_t ldab, double *dB, int64_t ldb, int32_t *d_info, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_trsv: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_trsv: kl out of [0, max(0, n-1)]");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_trsv: ku out of [0, max(0, n-1)]");
    BANDLU_ARG(kl == 0 || ku == 0, 3, "band_trsv: the band is not triangular (kl > 0 and ku > 0)");
    BANDLU_ARG(nrhs >= 0, 4, "band_trsv: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_trsv: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_trsv: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 7, "band_trsv: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 8, "band_trsv: ldb < max(1, n)");
    BANDLU_ARG(d_info != nullptr, 9, "band_trsv: d_info is null");
    if (n > kMaxN || nrhs > INT_MAX) {
        set_error("band_trsv: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return trsv(n, kl, ku, nrhs, dAB, ldab, ldab * n, dB, ldb, ldb * nrhs, d_info, 1,
                as_stream(stream));
}

extern "C" int band_trsv_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs,
                                 const double *dAB, int64_t ldab, int64_t strideAB, double *dB,
                                 int64_t ldb, int64_t strideB, int32_t *d_info, int64_t batch,
                                 void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_trsv_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_trsv_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_trsv_batched: ku out of range");
    BANDLU_ARG(kl == 0 || ku == 0, 3, "band_trsv_batched: the band is not triangular");
    BANDLU_ARG(nrhs >= 0, 4, "band_trsv_batched: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_trsv_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_trsv_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_trsv_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 8,
               "band_trsv_batched: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 9, "band_trsv_batched: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 10, "band_trsv_batched: strideB < ldb*nrhs");
    BANDLU_ARG(batch == 0 || d_info != nullptr, 11, "band_trsv_batched: d_info is null");
    BANDLU_ARG(batch >= 0, 12, "band_trsv_batched: batch < 0");
    if (n > kMaxN || batch > INT_MAX || nrhs > INT_MAX || batch * nrhs > INT_MAX) {
        set_error("band_trsv_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return trsv(n, kl, ku, nrhs, dAB, ldab, strideAB, dB, ldb, strideB, d_info, batch,
                as_stream(stream));
}

extern "C" int band_getrs_t(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                            int64_t ldab, const int32_t *d_ipiv, double *dB, int64_t ldb,
                            void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs_t: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs_t: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs_t: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs_t: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_getrs_t: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs_t: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || d_ipiv != nullptr, 7, "band_getrs_t: d_ipiv is null");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 8, "band_getrs_t: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 9, "band_getrs_t: ldb < max(1, n)");
    if (n > kMaxN || nrhs > INT_MAX) {
        set_error("band_getrs_t: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return getrs_t(n, kl, ku, nrhs, dAB, ldab, ldab * n, d_ipiv, n, dB, ldb, ldb * nrhs, 1,
                   as_stream(stream));
}

extern "C" int band_getrs_t_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs,
                                    const double *dAB, int64_t ldab, int64_t strideAB,
                                    const int32_t *d_ipiv, int64_t strideP, double *dB,
                                    int64_t ldb, int64_t strideB, int64_t batch, void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_getrs_t_batched: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_getrs_t_batched: kl out of range");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_getrs_t_batched: ku out of range");
    BANDLU_ARG(nrhs >= 0, 4, "band_getrs_t_batched: nrhs < 0");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 5, "band_getrs_t_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_getrs_t_batched: ldab < 2kl+ku+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 7, "band_getrs_t_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || d_ipiv != nullptr, 8,
               "band_getrs_t_batched: d_ipiv is null");
    BANDLU_ARG(batch <= 1 || strideP >= n, 9, "band_getrs_t_batched: strideP < n");
    BANDLU_ARG(n == 0 || nrhs == 0 || batch == 0 || dB != nullptr, 10,
               "band_getrs_t_batched: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 11, "band_getrs_t_batched: ldb < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideB >= ldb * nrhs, 12, "band_getrs_t_batched: strideB < ldb*nrhs");
    BANDLU_ARG(batch >= 0, 13, "band_getrs_t_batched: batch < 0");
    if (n > kMaxN || batch > INT_MAX || nrhs > INT_MAX || batch * nrhs > INT_MAX) {
        set_error("band_getrs_t_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return getrs_t(n, kl, ku, nrhs, dAB, ldab, strideAB, d_ipiv, strideP, dB, ldb, strideB, batch,
                   as_stream(stream));
}

// Factor and solve (xGBSV) as two calls with one dominant kernel each:
//   band_gbsv_lu:   band_getrf, and L y = P b on the right-hand sides (inside
//                   the persistent wide-band launch when that kernel runs, in
//                   a workgroup that trails the chain of panels; inside the
//                   lean window kernel's steps for one right-hand side when
//                   that kernel runs; else the forward chain after the
//                   factorisation);
//   band_gbsv_back: U x = y, the backward chain.
// band_gbsv is the two in turn.  The results are those of band_getrf and
// band_getrs, bitwise.
namespace bandlu {
namespace {
int gbsv_args(const char *fn, int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const void *dAB,
              int64_t ldab, const void *d_ipiv, const void *dB, int64_t ldb) {
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "%s: n < 0", fn);
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "%s: kl out of [0, max(0, n-1)]", fn);
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "%s: ku out of [0, max(0, n-1)]", fn);
    BANDLU_ARG(nrhs >= 0, 4, "%s: nrhs < 0", fn);
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "%s: dAB is null", fn);
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "%s: ldab < 2kl+ku+1", fn);
    BANDLU_ARG(n == 0 || d_ipiv != nullptr, 7, "%s: d_ipiv is null", fn);
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 8, "%s: dB is null", fn);
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 9, "%s: ldb < max(1, n)", fn);
    if (n > kMaxN || nrhs > INT_MAX) {
        set_error("%s: sizes too large", fn);
        return BANDLU_ERR_UNSUPPORTED;
    }
    return BANDLU_OK;
}
}  // namespace
}  // namespace bandlu

extern "C" int band_gbsv_lu(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, double *dAB,
                            int64_t ldab, int32_t *d_ipiv, double *dB, int64_t ldb,
                            int32_t *d_info, void *stream) {
    clear_error();
    if (int rc = gbsv_args("band_gbsv_lu", n, kl, ku, nrhs, dAB, ldab, d_ipiv, dB, ldb);
        rc != BANDLU_OK)
        return rc;
    BANDLU_ARG(d_info != nullptr, 10, "band_gbsv_lu: d_info is null");
    hipStream_t s = as_stream(stream);
    if (n > 0 && nrhs > 0 && band_getrf_variant(n, kl, ku, 1) == BANDLU_GETRF_WIDE &&
        getrf_wide_fused_fits(n, kl, ku, nrhs))
        return launch_getrf_wide(n, kl, ku, dAB, ldab, ldab * n, d_ipiv, n, d_info, 1, s, nullptr,
                                 0, dB, ldb, ldb * nrhs, nrhs);
    // one right-hand side and the lean window kernel: the forward solve runs
    // in the factorisation's own steps
    if (nrhs == 1) {
        const int rc = launch_getrf_lean_fwd(n, kl, ku, dAB, ldab, d_ipiv, dB, d_info, s);
        if (rc != BANDLU_ERR_UNSUPPORTED) return rc;
    }
    if (int rc = band_getrf(n, kl, ku, dAB, ldab, d_ipiv, d_info, stream); rc != BANDLU_OK)
        return rc;
    if (n < 2 || nrhs == 0 || kl == 0) return BANDLU_OK;
    RingParams P = chain_params(dAB, ldab, ldab * n, dB, ldb, ldb * nrhs, n, nrhs);
    P.ipiv = d_ipiv;
    P.strideP = n;
    P.kl = (int)kl;
    P.nsteps = (int)n - 1;
    P.cb0 = kl + ku;
    P.es = 1;
    P.K = (int)kl;
    return launch_chain(kRingFwdLU, P, 1, s);
}

extern "C" int band_gbsv_back(int64_t n, int64_t kl, int64_t ku, int64_t nrhs,
                              const double *dAB, int64_t ldab, double *dB, int64_t ldb,
                              void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 1, "band_gbsv_back: n < 0");
    BANDLU_ARG(kl >= 0 && kl <= bmax, 2, "band_gbsv_back: kl out of [0, max(0, n-1)]");
    BANDLU_ARG(ku >= 0 && ku <= bmax, 3, "band_gbsv_back: ku out of [0, max(0, n-1)]");
    BANDLU_ARG(nrhs >= 0, 4, "band_gbsv_back: nrhs < 0");
    BANDLU_ARG(n == 0 || dAB != nullptr, 5, "band_gbsv_back: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl + ku + 1, 6, "band_gbsv_back: ldab < 2kl+ku+1");
    BANDLU_ARG(n == 0 || nrhs == 0 || dB != nullptr, 7, "band_gbsv_back: dB is null");
    BANDLU_ARG(ldb >= (n > 1 ? n : 1), 8, "band_gbsv_back: ldb < max(1, n)");
    if (n > kMaxN || nrhs > INT_MAX) {
        set_error("band_gbsv_back: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    if (n == 0 || nrhs == 0) return BANDLU_OK;
    RingParams P = chain_params(dAB, ldab, ldab * n, dB, ldb, ldb * nrhs, n, nrhs);
    P.nsteps = (int)n;
    P.cb0 = 0;
    P.es = 1;
    P.K = (int)(kl + ku);
    return launch_chain(kRingBwd, P, 1, as_stream(stream));
}

extern "C" int band_gbsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, double *dAB,
                         int64_t ldab, int32_t *d_ipiv, double *dB, int64_t ldb, int32_t *d_info,
                         void *stream) {
    if (int rc = band_gbsv_lu(n, kl, ku, nrhs, dAB, ldab, d_ipiv, dB, ldb, d_info, stream);
        rc != BANDLU_OK)
        return rc;
    return band_gbsv_back(n, kl, ku, nrhs, dAB, ldab, dB, ldb, stream);
}
