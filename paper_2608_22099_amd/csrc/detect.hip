// Step 1 of the structure-aware strategy (Sec. II-A, cost I(N); Sec. III-A):
// find the lower and upper bandwidths of a dense column-major matrix.
//
// The scan is HBM-bound: every element is read once (8 bytes per element, one
// compare each).  Each wavefront owns a contiguous run of columns of the
// (batched) matrix, so it streams consecutive memory.  Within a column every
// lane reads 16 bytes per load (two rows) and several loads are in flight per
// lane; rows visited by one lane increase monotonically, so the first and last
// nonzero row of the lane's share of a column are kept with one compare and a
// select each.  Lane maxima of (last - j) and (j - first) are reduced across the
// wave once per matrix and published with one atomic max per value.
#include <climits>

#include <algorithm>

#include "common.hpp"

namespace bandlu {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;
typedef double dbl2 __attribute__((ext_vector_type(2)));

// Fused conversion: every element read that lies in the band of the caps,
// -pku <= i - j <= pkl, is also stored at AB[pkl + pku + i - j + j*ldab].
struct Pack {
    double *AB;
    int64_t ldab, strideAB;
    int pkl, pku;
};

template <bool PACK>
__device__ __forceinline__ void pack_store(const Pack &pk, int64_t b, int i, int c, double v) {
    if constexpr (PACK) {
        const int d = i - c;
        if (d >= -pk.pku && d <= pk.pkl)
            pk.AB[b * pk.strideAB + int64_t(pk.pkl + pk.pku + d) + int64_t(c) * pk.ldab] = v;
    }
}

struct DetectParams {
    const double *A;
    int64_t n, lda, strideA;
    int64_t total_cols;     // n * batch
    int64_t cols_per_wave;  // contiguous run of columns per wavefront
    int64_t kl_cap, ku_cap; // INT64_MAX when not capped
    unsigned long long *out;   // [3 * batch]
    unsigned long long *dmax;  // [3] or null
    Pack pk;
};

__global__ void detect_init(unsigned long long *out, int64_t count, unsigned long long *dmax) {
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i < count; i += int64_t(gridDim.x) * blockDim.x) out[i] = 0ull;
    if (dmax && blockIdx.x == 0 && threadIdx.x < 3) dmax[threadIdx.x] = 0ull;
}

// Batch maximum of the per-matrix results (one workgroup).
__global__ __launch_bounds__(kThreads) void detect_batch_max(const unsigned long long *out,
                                                             int64_t batch, unsigned long long *dmax) {
    int m0 = 0, m1 = 0, m2 = 0;
    for (int64_t b = threadIdx.x; b < batch; b += kThreads) {
        m0 = max(m0, int(out[3 * b + 0]));
        m1 = max(m1, int(out[3 * b + 1]));
        m2 = max(m2, int(out[3 * b + 2]));
    }
    __shared__ int s[3][kThreads / 64];
    m0 = wave_max_i32(m0);
    m1 = wave_max_i32(m1);
    m2 = wave_max_i32(m2);
    if ((threadIdx.x & 63) == 0) {
        s[0][threadIdx.x >> 6] = m0;
        s[1][threadIdx.x >> 6] = m1;
        s[2][threadIdx.x >> 6] = m2;
    }
    __syncthreads();
    if (threadIdx.x < 3) {
        int m = 0;
        for (int w = 0; w < kThreads / 64; ++w) m = max(m, s[threadIdx.x][w]);
        dmax[threadIdx.x] = (unsigned long long)m;
    }
}

// Raise *p to v.  Atomics on one address serialise in L2, and most
// workgroups hold a value that is already published, so read first and issue
// the atomic only when it can change the result.
__device__ inline bool publish_max(unsigned long long *p, unsigned long long v) {
    if (v > __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        atomicMax(p, v);
        return true;
    }
    return false;
}

// Publish the wave's bandwidths of matrix b.
__device__ inline void detect_flush(const DetectParams &P, int64_t b, int kl_l, int ku_l, int lane) {
    int kl_w = wave_max_i32(kl_l);
    int ku_w = wave_max_i32(ku_l);
    if (lane == 0) {
        unsigned long long *o = P.out + 3 * b;
        const bool r0 = publish_max(o + 0, (unsigned long long)kl_w);
        const bool r1 = publish_max(o + 1, (unsigned long long)ku_w);
        const bool ex = (int64_t)kl_w > P.kl_cap || (int64_t)ku_w > P.ku_cap;
        const bool r2 = ex && publish_max(o + 2, 1ull);
        if (P.dmax) {
            if (r0) publish_max(P.dmax + 0, (unsigned long long)kl_w);
            if (r1) publish_max(P.dmax + 1, (unsigned long long)ku_w);
            if (r2) publish_max(P.dmax + 2, 1ull);
        }
    }
}

template <bool VEC, bool CAPS, bool PACK>
__global__ __launch_bounds__(kThreads) void detect_kernel(DetectParams P) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t(blockIdx.x) * kThreads + threadIdx.x) >> 6;
    const int64_t g0 = wave * P.cols_per_wave;
    const int64_t g1 = min(g0 + P.cols_per_wave, P.total_cols);
    if (g0 >= g1) return;
    const int64_t n = P.n;
    int64_t b = g0 / n;
    int64_t j = g0 - b * n;
    int kl_l = 0, ku_l = 0;
    bool skip = false;  // matrix b already known to exceed a cap
    for (int64_t g = g0; g < g1; ++g) {
        if (CAPS && !skip) {
            skip = __hip_atomic_load(P.out + 3 * b + 2, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) != 0ull;
        }
        if (!skip) {
            const double *col = P.A + b * P.strideA + j * P.lda;
            int first = INT_MAX, last = -1;
            if (VEC) {
                const dbl2 *c2 = reinterpret_cast<const dbl2 *>(col);
                const int n2 = int(n >> 1);
                for (int base = 0; base < n2; base += 64 * kUnroll) {
                    // (rows 2base..2base+128kUnroll-1 meet the caps' band?)
                    const bool pk_here = PACK && 2 * base <= int(j) + P.pk.pkl &&
                                         2 * (base + 64 * kUnroll) - 1 >= int(j) - P.pk.pku;
                    dbl2 v[kUnroll];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        int idx = base + u * 64 + lane;
                        v[u] = idx < n2 ? __builtin_nontemporal_load(c2 + idx) : dbl2{0.0, 0.0};
                    }
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        int i0 = 2 * (base + u * 64 + lane);
                        if (v[u].x != 0.0) { last = i0; first = min(first, i0); }
                        if (v[u].y != 0.0) { last = i0 + 1; first = min(first, i0 + 1); }
                        if (pk_here && base + u * 64 + lane < n2) {
                            pack_store<PACK>(P.pk, b, i0, int(j), v[u].x);
                            pack_store<PACK>(P.pk, b, i0 + 1, int(j), v[u].y);
                        }
                    }
                }
                if ((n & 1) && lane == 0) {
                    int i0 = int(n - 1);
                    if (col[i0] != 0.0) { last = i0; first = min(first, i0); }
                    pack_store<PACK>(P.pk, b, i0, int(j), col[i0]);
                }
            } else {
                const int nn = int(n);
                for (int base = 0; base < nn; base += 64 * kUnroll) {
                    const bool pk_here = PACK && base <= int(j) + P.pk.pkl &&
                                         base + 64 * kUnroll - 1 >= int(j) - P.pk.pku;
                    double v[kUnroll];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        int idx = base + u * 64 + lane;
                        v[u] = idx < nn ? __builtin_nontemporal_load(col + idx) : 0.0;
                    }
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        int i0 = base + u * 64 + lane;
                        if (v[u] != 0.0) { last = i0; first = min(first, i0); }
                        if (pk_here && i0 < nn) pack_store<PACK>(P.pk, b, i0, int(j), v[u]);
                    }
                }
            }
            const int jj = int(j);
            if (last >= 0) {
                kl_l = max(kl_l, last - jj);
                ku_l = max(ku_l, jj - first);
            }
            if (CAPS) {
                bool ex = (int64_t)kl_l > P.kl_cap || (int64_t)ku_l > P.ku_cap;
                // tell every other wave of this matrix to stop early
                if (__any(ex) && lane == 0)
                    __hip_atomic_store(P.out + 3 * b + 2, 1ull, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (++j == n) {
            detect_flush(P, b, kl_l, ku_l, lane);
            kl_l = ku_l = 0;
            skip = false;
            j = 0;
            ++b;
        }
    }
    if (j != 0) detect_flush(P, b, kl_l, ku_l, lane);
}

// Contiguous matrices (lda == n): the data is one flat stream cut into 32 KiB
// chunks that consecutive workgroups take in turn, so the whole chip reads one
// contiguous front of memory.
//   single matrix (BATCHED = false): n even and >= 2048, so a chunk spans at
//     most three columns; maxima are kept across chunks and published once;
//   batch (BATCHED = true): n a power of two with n*n a multiple of the chunk,
//     so a chunk lies in one matrix; each wave publishes per chunk.
// n even keeps both doubles of a 16-byte load in one column.
constexpr int kFlatU = 8;
constexpr int kFlatChunk = kThreads * 2 * kFlatU;  // doubles per chunk

struct FlatParams {
    const double *A;
    int64_t n, total, nchunks;
    int64_t kl_cap, ku_cap;
    unsigned long long *out;   // [3 * batch]
    unsigned long long *dmax;  // [3] (batched) or null
    int64_t chunks_per_matrix; // batched: n*n / kFlatChunk
    int log2n;                 // batched: n = 2^log2n
    Pack pk;
};

template <bool CAPS, bool BATCHED, bool PACK>
__global__ __launch_bounds__(kThreads) void detect_flat_kernel(FlatParams P) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int n = int(P.n);
    int kl_t = 0, ku_t = 0;
    // the loads of a workgroup's next chunk are issued before it scans the
    // current one, so that its reads stay in flight across chunks
    auto load = [&](int64_t k, dbl2 *v) __attribute__((always_inline)) {
        const int64_t f0 = k * kFlatChunk;
        const dbl2 *base = reinterpret_cast<const dbl2 *>(P.A + f0);
#pragma unroll
        for (int u = 0; u < kFlatU; ++u) {
            const int e = u * (kThreads * 2) + tid * 2;
            v[u] = f0 + e < P.total ? __builtin_nontemporal_load(base + (e >> 1)) : dbl2{0.0, 0.0};
        }
    };
    dbl2 v[kFlatU], vn[kFlatU];
    if (int64_t(blockIdx.x) < P.nchunks) load(blockIdx.x, v);
    for (int64_t k = blockIdx.x; k < P.nchunks; k += gridDim.x) {
        const int64_t mat = BATCHED ? k / P.chunks_per_matrix : 0;
        unsigned long long *out = P.out + 3 * mat;
        if (k + gridDim.x < P.nchunks) load(k + gridDim.x, vn);
        if (CAPS && __hip_atomic_load(out + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0ull) {
            if (BATCHED) {
#pragma unroll
                for (int u = 0; u < kFlatU; ++u) v[u] = vn[u];
                continue;
            }
            break;
        }
        const int64_t f0 = k * kFlatChunk;
        const int64_t fm = BATCHED ? f0 - mat * P.n * P.n : f0;  // offset inside the matrix
        // the chunk [fm, fm + chunk) meets the caps' band, i.e. some column c
        // has c (n+1) in [fm - pkl, fm + chunk - 1 + pku] (element (i, c) is at
        // c n + i, and -pku <= i - c <= pkl)
        bool pk_here = false;
        if constexpr (PACK) {
            const int64_t lo = fm - P.pk.pkl, hi = fm + kFlatChunk - 1 + P.pk.pku;
            const int64_t np1 = P.n + 1;
            const int64_t clo = lo <= 0 ? 0 : (lo + np1 - 1) / np1;
            const int64_t chi = hi / np1;
            pk_here = clo <= chi;
        }
        const int64_t col0 = BATCHED ? (fm >> P.log2n) : fm / P.n;
        const int i0 = int(fm - col0 * P.n);
        const int c0 = int(col0);
#pragma unroll
        for (int u = 0; u < kFlatU; ++u) {
            const int e = u * (kThreads * 2) + tid * 2;
            int i = i0 + e, c = c0;
            if (BATCHED) {
                c += i >> P.log2n;
                i &= n - 1;
            } else {
                while (i >= n) {  // n >= 2048: at most two wraps per 4096-element chunk
                    i -= n;
                    ++c;
                }
            }
            const int d = i - c;
            if (v[u].x != 0.0) { kl_t = max(kl_t, d); ku_t = max(ku_t, -d); }
            if (v[u].y != 0.0) { kl_t = max(kl_t, d + 1); ku_t = max(ku_t, -d - 1); }
            if (pk_here && f0 + e < P.total) {
                pack_store<PACK>(P.pk, mat, i, c, v[u].x);
                pack_store<PACK>(P.pk, mat, i + 1, c, v[u].y);
            }
        }
#pragma unroll
        for (int u = 0; u < kFlatU; ++u) v[u] = vn[u];
        if (BATCHED) {
            const int a = wave_max_i32(kl_t), b = wave_max_i32(ku_t);
            if (lane == 0) {
                // non-returning atomics: the wave goes on to its next chunk
                // without waiting; the batch maximum is formed afterwards
                if (a > 0) atomicMax(out + 0, (unsigned long long)a);
                if (b > 0) atomicMax(out + 1, (unsigned long long)b);
                if ((int64_t)a > P.kl_cap || (int64_t)b > P.ku_cap) atomicMax(out + 2, 1ull);
            }
            kl_t = ku_t = 0;
        } else if (CAPS) {
            const bool ex = (int64_t)kl_t > P.kl_cap || (int64_t)ku_t > P.ku_cap;
            if (__any(ex) && lane == 0)
                __hip_atomic_store(out + 2, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (BATCHED) return;
    __shared__ int s_kl[kThreads / 64], s_ku[kThreads / 64];
    kl_t = wave_max_i32(kl_t);
    ku_t = wave_max_i32(ku_t);
    if (lane == 0) { s_kl[tid >> 6] = kl_t; s_ku[tid >> 6] = ku_t; }
    __syncthreads();
    if (tid == 0) {
        int a = 0, b = 0;
        for (int w = 0; w < kThreads / 64; ++w) { a = max(a, s_kl[w]); b = max(b, s_ku[w]); }
        publish_max(P.out + 0, (unsigned long long)a);
        publish_max(P.out + 1, (unsigned long long)b);
        if ((int64_t)a > P.kl_cap || (int64_t)b > P.ku_cap) publish_max(P.out + 2, 1ull);
    }
}

// After a fused pass: the band of the detected (kl, ku) (batched: the batch
// maximum) starts pkl + pku - kl - ku rows into each matrix's band array.
// Write +0.0 into that view's fill rows (0..kl-1) and into its slots outside
// the matrix, as the conversion step does; nothing when a cap was exceeded.
__global__ __launch_bounds__(256) void pack_fixup_kernel(Pack pk, int64_t n, int64_t batch,
                                                         const unsigned long long *klku) {
    if (klku[2] != 0ull) return;
    const int64_t kl = int64_t(klku[0]), ku = int64_t(klku[1]);
    const int64_t shift = pk.pkl + pk.pku - kl - ku;
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
    const int64_t waves = (int64_t(gridDim.x) * blockDim.x) >> 6;
    // one wavefront per column: its fill rows 0..kl-1, and the rows of its
    // slots above row 0 (c < ku) or below row n-1 (c > n-1-kl)
    for (int64_t bc = wave; bc < batch * n; bc += waves) {
        const int64_t c = bc % n, b = bc / n;
        double *col = pk.AB + b * pk.strideAB + shift + c * pk.ldab;
        const int64_t top = kl + (c < ku ? ku - c : 0);           // rows [0, top): fill or i < 0
        const int64_t bot = kl + ku + (n - c);                     // rows [bot, 2kl+ku]: i >= n
        for (int64_t r = lane; r < top; r += 64) col[r] = 0.0;
        for (int64_t r = bot + lane; r <= 2 * kl + ku; r += 64) col[r] = 0.0;
    }
}

int launch_detect(const double *dA, int64_t n, int64_t lda, int64_t strideA, int64_t batch,
                  int64_t kl_cap, int64_t ku_cap, int64_t *d_out, int64_t *d_max,
                  hipStream_t s, const Pack *pack = nullptr) {
    const int64_t count = 3 * batch;
    {
        int blocks = (int)std::min<int64_t>((count + 255) / 256, 1024);
        if (blocks < 1) blocks = 1;
        hipLaunchKernelGGL(detect_init, dim3(blocks), dim3(256), 0, s,
                           reinterpret_cast<unsigned long long *>(d_out), count,
                           reinterpret_cast<unsigned long long *>(d_max));
        BANDLU_CHECK_LAUNCH("band_detect init");
    }
    if (n == 0 || batch == 0) return BANDLU_OK;
    const bool caps = kl_cap >= 0 || ku_cap >= 0;
    const bool pk = pack != nullptr;
    const Pack pkv = pk ? *pack : Pack{};
    const bool aligned = reinterpret_cast<uintptr_t>(dA) % 16 == 0;
    int log2n = 0;
    while ((int64_t(1) << log2n) < n) ++log2n;
    const bool single_flat = batch == 1 && lda == n && n % 2 == 0 && n >= 2048 && aligned;
    const bool batch_flat = batch > 1 && lda == n && strideA == n * n && (int64_t(1) << log2n) == n &&
                            (n * n) % kFlatChunk == 0 && aligned;
    if (single_flat || batch_flat) {
        FlatParams F;
        F.A = dA;
        F.n = n;
        F.total = n * n * batch;
        F.nchunks = (F.total + kFlatChunk - 1) / kFlatChunk;
        F.kl_cap = kl_cap < 0 ? INT64_MAX : kl_cap;
        F.ku_cap = ku_cap < 0 ? INT64_MAX : ku_cap;
        F.out = reinterpret_cast<unsigned long long *>(d_out);
        F.dmax = reinterpret_cast<unsigned long long *>(d_max);
        F.chunks_per_matrix = (n * n) / kFlatChunk;
        F.log2n = log2n;
        F.pk = pkv;
        const int64_t grid = std::min<int64_t>(F.nchunks, int64_t(device_cu_count()) * 8);
        auto k = pk ? (single_flat ? detect_flat_kernel<true, false, true> : detect_flat_kernel<true, true, true>)
                 : single_flat ? (caps ? detect_flat_kernel<true, false, false> : detect_flat_kernel<false, false, false>)
                               : (caps ? detect_flat_kernel<true, true, false> : detect_flat_kernel<false, true, false>);
        hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kThreads), 0, s, F);
        BANDLU_CHECK_LAUNCH("band_detect (flat)");
        // the batch maximum (also for a batch of one that took the
        // single-matrix kernel, which publishes to d_out only)
        if (batch_flat || d_max != nullptr) {
            hipLaunchKernelGGL(detect_batch_max, dim3(1), dim3(kThreads), 0, s,
                               reinterpret_cast<const unsigned long long *>(d_out), batch,
                               reinterpret_cast<unsigned long long *>(d_max));
            BANDLU_CHECK_LAUNCH("band_detect (batch max)");
        }
        return BANDLU_OK;
    }
    DetectParams P;
    P.A = dA;
    P.n = n;
    P.lda = lda;
    P.strideA = strideA;
    P.total_cols = n * batch;
    const int64_t max_waves = int64_t(device_cu_count()) * 32;  // 8 waves per SIMD
    const int64_t waves = std::min(P.total_cols, max_waves);
    P.cols_per_wave = (P.total_cols + waves - 1) / waves;
    const int64_t used_waves = (P.total_cols + P.cols_per_wave - 1) / P.cols_per_wave;
    const int64_t blocks = (used_waves + (kThreads / 64) - 1) / (kThreads / 64);
    P.kl_cap = kl_cap < 0 ? INT64_MAX : kl_cap;
    P.ku_cap = ku_cap < 0 ? INT64_MAX : ku_cap;
    P.out = reinterpret_cast<unsigned long long *>(d_out);
    P.dmax = reinterpret_cast<unsigned long long *>(d_max);
    P.pk = pkv;
    const bool vec = (reinterpret_cast<uintptr_t>(dA) % 16 == 0) && (lda % 2 == 0) &&
                     (batch == 1 || strideA % 2 == 0);
    auto k = pk ? (vec ? detect_kernel<true, true, true> : detect_kernel<false, true, true>)
           : vec ? (caps ? detect_kernel<true, true, false> : detect_kernel<true, false, false>)
                 : (caps ? detect_kernel<false, true, false> : detect_kernel<false, false, false>);
    hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(kThreads), 0, s, P);
    BANDLU_CHECK_LAUNCH("band_detect");
    return BANDLU_OK;
}

}  // namespace
}  // namespace bandlu

using namespace bandlu;

extern "C" int band_detect(const double *dA, int64_t n, int64_t lda, int64_t kl_cap,
                           int64_t ku_cap, int64_t *d_out, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 2, "band_detect: n = %lld < 0", (long long)n);
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "band_detect: lda = %lld < max(1, n)", (long long)lda);
    BANDLU_ARG(d_out != nullptr, 6, "band_detect: d_out is null");
    BANDLU_ARG(n == 0 || dA != nullptr, 1, "band_detect: dA is null");
    if (n > kMaxN) {
        set_error("band_detect: n >= 2^31 is not supported");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_detect(dA, n, lda, lda * n, 1, kl_cap, ku_cap, d_out, nullptr,
                         as_stream(stream));
}

extern "C" int band_detect_batched(const double *dA, int64_t n, int64_t lda, int64_t strideA,
                                   int64_t batch, int64_t kl_cap, int64_t ku_cap,
                                   int64_t *d_out, int64_t *d_max, void *stream) {
    clear_error();
    BANDLU_ARG(n >= 0, 2, "band_detect_batched: n = %lld < 0", (long long)n);
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "band_detect_batched: lda < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideA >= lda * n, 4, "band_detect_batched: strideA < lda*n");
    BANDLU_ARG(batch >= 0, 5, "band_detect_batched: batch < 0");
    BANDLU_ARG(batch == 0 || d_out != nullptr, 8, "band_detect_batched: d_out is null");
    BANDLU_ARG(d_max != nullptr, 9, "band_detect_batched: d_max is null");
    BANDLU_ARG(n == 0 || batch == 0 || dA != nullptr, 1, "band_detect_batched: dA is null");
    if (n > kMaxN || (n > 0 && batch > INT64_MAX / n)) {
        set_error("band_detect_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return launch_detect(dA, n, lda, strideA, batch, kl_cap, ku_cap, d_out, d_max,
                         as_stream(stream));
}

// ------------------------------------------------ fused detect + convert --
// Steps 1 and 2 in one read of the dense matrix (Sec. II-A: I(N) and C(N);
// Listing 2's detection and conversion): detection under the caps, and every
// element inside the caps' band stored into a band array laid out for the
// caps; then the fix-up above.
namespace bandlu {
namespace {
int detect_convert(const double *dA, int64_t n, int64_t lda, int64_t strideA, int64_t batch,
                   int64_t kl_cap, int64_t ku_cap, int64_t *d_out, int64_t *d_max, double *dAB,
                   int64_t ldab, int64_t strideAB, hipStream_t s) {
    Pack pk;
    pk.AB = dAB;
    pk.ldab = ldab;
    pk.strideAB = strideAB;
    pk.pkl = (int)kl_cap;
    pk.pku = (int)ku_cap;
    if (int rc = launch_detect(dA, n, lda, strideA, batch, kl_cap, ku_cap, d_out, d_max, s, &pk);
        rc != BANDLU_OK)
        return rc;
    if (n == 0 || batch == 0) return BANDLU_OK;
    const int64_t total = batch * n * 64;  // a wavefront per column
    const unsigned grid = (unsigned)std::min<int64_t>((total + 255) / 256, int64_t(device_cu_count()) * 16);
    hipLaunchKernelGGL(pack_fixup_kernel, dim3(grid), dim3(256), 0, s, pk, n, batch,
                       reinterpret_cast<const unsigned long long *>(batch == 1 && d_max == nullptr ? d_out : d_max));
    BANDLU_CHECK_LAUNCH("band_detect_convert (fix-up)");
    return BANDLU_OK;
}
}  // namespace
}  // namespace bandlu

extern "C" int band_detect_convert(const double *dA, int64_t n, int64_t lda, int64_t kl_cap,
                                   int64_t ku_cap, int64_t *d_out, double *dAB, int64_t ldab,
                                   void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 2, "band_detect_convert: n = %lld < 0", (long long)n);
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "band_detect_convert: lda < max(1, n)");
    BANDLU_ARG(kl_cap >= 0 && kl_cap <= bmax, 4, "band_detect_convert: kl_cap out of [0, max(0, n-1)]");
    BANDLU_ARG(ku_cap >= 0 && ku_cap <= bmax, 5, "band_detect_convert: ku_cap out of [0, max(0, n-1)]");
    BANDLU_ARG(d_out != nullptr, 6, "band_detect_convert: d_out is null");
    BANDLU_ARG(n == 0 || dAB != nullptr, 7, "band_detect_convert: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl_cap + ku_cap + 1, 8, "band_detect_convert: ldab < 2kl_cap+ku_cap+1");
    BANDLU_ARG(n == 0 || dA != nullptr, 1, "band_detect_convert: dA is null");
    if (n > kMaxN || n * ldab > (int64_t(1) << 40)) {
        set_error("band_detect_convert: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return detect_convert(dA, n, lda, lda * n, 1, kl_cap, ku_cap, d_out, nullptr, dAB, ldab,
                          ldab * n, as_stream(stream));
}

extern "C" int band_detect_convert_batched(const double *dA, int64_t n, int64_t lda,
                                           int64_t strideA, int64_t batch, int64_t kl_cap,
                                           int64_t ku_cap, int64_t *d_out, int64_t *d_max,
                                           double *dAB, int64_t ldab, int64_t strideAB,
                                           void *stream) {
    clear_error();
    const int64_t bmax = n > 1 ? n - 1 : 0;
    BANDLU_ARG(n >= 0, 2, "band_detect_convert_batched: n < 0");
    BANDLU_ARG(lda >= (n > 1 ? n : 1), 3, "band_detect_convert_batched: lda < max(1, n)");
    BANDLU_ARG(batch <= 1 || strideA >= lda * n, 4, "band_detect_convert_batched: strideA < lda*n");
    BANDLU_ARG(batch >= 0, 5, "band_detect_convert_batched: batch < 0");
    BANDLU_ARG(kl_cap >= 0 && kl_cap <= bmax, 6, "band_detect_convert_batched: kl_cap out of range");
    BANDLU_ARG(ku_cap >= 0 && ku_cap <= bmax, 7, "band_detect_convert_batched: ku_cap out of range");
    BANDLU_ARG(batch == 0 || d_out != nullptr, 8, "band_detect_convert_batched: d_out is null");
    BANDLU_ARG(d_max != nullptr, 9, "band_detect_convert_batched: d_max is null");
    BANDLU_ARG(n == 0 || batch == 0 || dAB != nullptr, 10, "band_detect_convert_batched: dAB is null");
    BANDLU_ARG(ldab >= 2 * kl_cap + ku_cap + 1, 11,
               "band_detect_convert_batched: ldab < 2kl_cap+ku_cap+1");
    BANDLU_ARG(batch <= 1 || strideAB >= ldab * n, 12,
               "band_detect_convert_batched: strideAB < ldab*n");
    BANDLU_ARG(n == 0 || batch == 0 || dA != nullptr, 1, "band_detect_convert_batched: dA is null");
    if (n > kMaxN || (n > 0 && batch > INT64_MAX / n)) {
        set_error("band_detect_convert_batched: sizes too large");
        return BANDLU_ERR_UNSUPPORTED;
    }
    return detect_convert(dA, n, lda, strideA, batch, kl_cap, ku_cap, d_out, d_max, dAB, ldab,
                          strideAB, as_stream(stream));
}
