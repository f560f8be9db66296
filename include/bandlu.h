/*
 * bandlu.h -- C ABI of libbandlu.so: the structure-aware banded LU path of
 * "When Structure is Silent: Opportunities for Algorithmic Dispatch in Linear
 * Algebra" on AMD Instinct MI355X (gfx950).
 *
 * The paper's strategy (Sec. II-A) has three steps: identify the structure of
 * a dense-stored N x N matrix, convert it to a structure-specific format, and
 * apply the specialised algorithm.  For LU of banded matrices (Sec. III,
 * Listing 2) these are: detect the bandwidths, pack into the xGBTRF band
 * layout, and run banded LU with partial pivoting (xGBTRF); the factors then
 * solve A x = b (the backslash of Listing 1).  Each entry point below is one
 * of these steps, run by hand-written HIP kernels.
 *
 * Common conventions
 *   - Precision: IEEE binary64 throughout.
 *   - Dense matrices are column-major: element (i, j), 0-based, at
 *     A[i + j*lda], lda >= max(1, n).  Rows n..lda-1 of a column are never read.
 *   - Band storage is the LAPACK xGBTRF layout: element (i, j) at
 *     AB[kl + ku + i - j + j*ldab] for max(0, j-ku) <= i <= min(n-1, j+kl),
 *     ldab >= 2*kl + ku + 1.  Band rows 0..kl-1 hold the fill-in that row
 *     interchanges create in U (U has kl+ku superdiagonals).
 *   - Pointers prefixed d are device pointers (HBM of the current device);
 *     all buffers are owned and allocated by the caller.  The library keeps
 *     no allocation between calls, frees nothing and holds no global state
 *     other than a thread-local text of the last error.
 *   - stream is a hipStream_t (NULL = the legacy default stream).  Every call
 *     only enqueues work on that stream and returns; results are valid after
 *     the stream is synchronised.  No entry point synchronises or copies to
 *     the host.
 *   - Batched calls take a stride (in elements) between consecutive matrices,
 *     pivot vectors and right-hand-side blocks.
 *   - Sizes are int64; n must be < 2^31 (pivot indices are int32).
 *
 * Return status
 *    0                 success (work enqueued)
 *   -k  (k >= 1)       argument k (1-based, in declaration order) is invalid;
 *                      nothing was enqueued
 *   BANDLU_ERR_HIP     a HIP runtime call or kernel launch failed
 *   BANDLU_ERR_UNSUPPORTED  the arguments are valid but beyond what the
 *                      library implements (e.g. n >= 2^31)
 * band_status_string() names a status; band_last_error() gives details of the
 * last failure on the calling thread.
 */
#ifndef BANDLU_H
#define BANDLU_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BANDLU_OK 0
#define BANDLU_ERR_HIP (-1000)
#define BANDLU_ERR_UNSUPPORTED (-1001)

/*
 * band_detect -- step 1, identify the structure (Sec. II-A cost I(N);
 * Sec. III-A: an O(N^2) scan; Listing 2 banded-structure test; Listing 1
 * decides triangularity by inspecting the elements the same way).
 *
 * Scans the dense n x n matrix dA (column-major, leading dimension lda) and
 * writes to device memory d_out[0..2] (int64):
 *   d_out[0] = kl = max(0, max of i - j over entries with A(i,j) != 0.0)
 *   d_out[1] = ku = max(0, max of j - i over entries with A(i,j) != 0.0)
 *   d_out[2] = 1 if (kl_cap >= 0 and kl > kl_cap) or (ku_cap >= 0 and
 *              ku > ku_cap), else 0.
 * "!= 0.0" is the IEEE comparison: -0.0 counts as zero, NaN/Inf/subnormals as
 * nonzero.  A cap < 0 means no cap.  With a cap set, the scan may stop early
 * once a bandwidth is known to exceed it; then d_out[2] = 1 and d_out[0..1]
 * are lower bounds of the true bandwidths, at least one of them above its
 * cap.  Whenever d_out[2] = 0 the bandwidths are exact.  n = 0 writes
 * {0, 0, 0}.  d_out must be 8-byte aligned; it is overwritten.
 */
int band_detect(const double *dA, int64_t n, int64_t lda, int64_t kl_cap, int64_t ku_cap,
                int64_t *d_out, void *stream);

/*
 * band_detect_batched -- step 1 (Sec. II-A cost I(N), Sec. III-A) over
 * many independent systems: band_detect over `batch` matrices of the same n;
 * matrix b starts at dA + b*strideA (strideA >= lda*n).  Writes
 * d_out[3b..3b+2] per matrix as band_detect does, and d_max[0..2] =
 * {max kl, max ku, any exceeded} over the batch (the bandwidths a single
 * uniform band layout for the whole batch needs).
 */
int band_detect_batched(const double *dA, int64_t n, int64_t lda, int64_t strideA,
                        int64_t batch, int64_t kl_cap, int64_t ku_cap, int64_t *d_out,
                        int64_t *d_max, void *stream);

/*
 * dense_to_band -- step 2, convert (Sec. II-A cost C(N); Listing 2 converts
 * the dense matrix to a band matrix before the banded LU).
 *
 * Writes rows 0..2kl+ku of the n columns of dAB (xGBTRF layout, leading
 * dimension ldab): every in-band element of A is copied bit for bit (so -0.0
 * and NaN payloads survive); every other slot of those rows -- the kl fill
 * rows and the corners outside the matrix -- becomes +0.0.  Rows >= 2kl+ku+1
 * of dAB are not touched.  Entries of A outside the band (kl, ku) are
 * ignored.  0 <= kl, ku <= max(0, n-1).  dA and dAB must not overlap.
 */
int dense_to_band(const double *dA, int64_t n, int64_t lda, int64_t kl, int64_t ku,
                  double *dAB, int64_t ldab, void *stream);

/*
 * dense_to_band_batched -- step 2 (Sec. II-A cost C(N); Listing 2's
 * conversion) over many independent systems: dense_to_band for `batch`
 * matrices: matrix b at
 * dA + b*strideA, its band at dAB + b*strideAB (strideAB >= ldab*n).
 */
int dense_to_band_batched(const double *dA, int64_t n, int64_t lda, int64_t strideA,
                          int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                          int64_t strideAB, int64_t batch, void *stream);

/*
 * band_getrf -- step 3, the specialised algorithm (Sec. II-A cost f(N);
 * Sec. III-A: banded LU, xGBTRF, O(N P Q)).  LU factorisation with partial
 * pivoting of the n x n band matrix in dAB (xGBTRF layout), in place, with
 * xGBTRF semantics:
 *   - on entry rows kl..2kl+ku of dAB hold A; rows 0..kl-1 need not be set
 *     and are never read (the routine zeroes the in-matrix fill slots);
 *   - on exit rows 0..kl+ku hold U (kl+ku superdiagonals) and rows
 *     kl+ku+1..2kl+ku the multipliers of L, unpermuted (product form);
 *     slots outside the matrix are not written;
 *   - d_ipiv[j] (int32, 1-based): row j was interchanged with row
 *     d_ipiv[j]-1.  The pivot is the first entry of largest magnitude in the
 *     column (BLAS i_amax: a NaN is taken only in first position);
 *   - *d_info (int32) = 0, or j+1 for the first exactly-zero pivot in 0-based
 *     column j; the factorisation still completes, as in xGBTRF.
 * Multipliers are formed as a * (1/pivot) when |pivot| >= DBL_MIN, else as
 * a / pivot; every update is one fused multiply-add.  Below the
 * dense-contraction threshold (kl < 32) the factors are bitwise those of the
 * unblocked algorithm on finite data.  From kl = 32 on (and kl <= 256) each
 * panel of 32 columns is applied to the rest of the band as a dense product
 * on the fp64 matrix cores, in one persistent launch (BANDLU_GETRF_WIDE)
 * when the batch fits the device's co-resident workgroups; each entry still
 * receives its fused multiply-adds in the order of the column steps, and the
 * factors are compared with the unblocked ones to a relative 1e-10.  The
 * persistent launch allocates its hand-off scratch (about 75 KB per 32
 * columns of kl+ku, per matrix) stream-ordered on `stream` and frees it the
 * same way; its workgroups wait for each other with bounded waits, and if a
 * wait ever ran out the kernel stops and sets *d_info = INT_MIN (the factors
 * are then invalid).
 */
int band_getrf(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab, int32_t *d_ipiv,
               int32_t *d_info, void *stream);

/*
 * band_getrf_batched -- step 3 (Sec. II-A cost f(N); Sec. III-A banded LU,
 * xGBTRF) over many independent systems: band_getrf on `batch` independent
 * matrices of the same
 * n, kl, ku: band b at dAB + b*strideAB (strideAB >= ldab*n), pivots at
 * d_ipiv + b*strideP (strideP >= n), info at d_info[b].
 */
int band_getrf_batched(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                       int64_t strideAB, int32_t *d_ipiv, int64_t strideP, int32_t *d_info,
                       int64_t batch, void *stream);

/*
 * band_getrf_batched_noalloc -- band_getrf_batched for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Arguments, results and the kernel chosen
 * are those of band_getrf_batched, and so the factors, ipiv and info are
 * bitwise the same.  The caller still owns dAB, d_ipiv and d_info.  The one
 * kernel that needs scratch, the persistent wide-band one, takes its
 * hand-off ring from a fixed 16 MiB array that the library holds on each
 * device it runs on until the process ends.  The function itself calls no
 * hipMalloc, hipFree or other allocating routine.
 *   - A matrix whose ring would exceed 16 MiB is rejected with
 *     BANDLU_ERR_UNSUPPORTED before anything is enqueued.  Such a matrix has
 *     kl >= 32 and kl+ku above about 7100; for kl = ku = 256 the ring is about
 *     1.3 MB per matrix.
 *   - A batch is factored in as many launches as the array needs, one after
 *     another on `stream`.
 *   - The first call on a device looks up the array's address on that device
 *     (the current one).  `stream` must belong to that device.
 *   - Every call on one device shares that device's array, and it keeps the
 *     last call's contents (each launch clears its own counters first).  Calls
 *     that overlap on one device race: calls on different streams, or from
 *     different threads without ordering, corrupt each other's factors.
 */
int band_getrf_batched_noalloc(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                               int64_t strideAB, int32_t *d_ipiv, int64_t strideP,
                               int32_t *d_info, int64_t batch, void *stream);

/*
 * band_getrs -- solve A X = B with the factors from band_getrf (the "lu(A) \
 * B" of Listings 1 and 2; xGBTRS, no transpose).  dB is n x nrhs,
 * column-major, leading dimension ldb >= max(1, n), overwritten with X.
 *   forward:  for j = 0..n-2: swap b[j], b[ipiv[j]-1];
 *             b[j+t] = fma(-l_t, b[j], b[j+t]) for t = 1..min(kl, n-1-j)
 *   backward: for j = n-1..0: b[j] = b[j] / U(j,j);
 *             b[i] = fma(-U(i,j), b[j], b[i]) for max(0, j-kl-ku) <= i < j
 * The result is bitwise that of this sequence.  A zero U(j,j) (info > 0)
 * yields Inf/NaN, as in xGBTRS.
 */
int band_getrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB, int64_t ldab,
               const int32_t *d_ipiv, double *dB, int64_t ldb, void *stream);

/*
 * band_getrs_batched -- the solve of Listings 1 and 2 ("lu(A) \ B", xGBTRS)
 * over many independent systems: band_getrs on `batch` systems: factors at
 * dAB + b*strideAB, pivots at d_ipiv + b*strideP, right-hand sides at
 * dB + b*strideB (strideB >= ldb*nrhs).
 */
int band_getrs_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                       int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                       double *dB, int64_t ldb, int64_t strideB, int64_t batch, void *stream);

/*
 * band_getrf_variant -- which factorisation kernel band_getrf(_batched) runs
 * for these sizes (host-only, enqueues nothing).  Returns one of the
 * BANDLU_GETRF_* codes below, or a negative status for invalid sizes.
 */
#define BANDLU_GETRF_WINDOW 1       /* register window, 64 lanes per matrix     */
#define BANDLU_GETRF_WINDOW_G16 2   /* register window, 16 lanes per matrix     */
#define BANDLU_GETRF_GENERIC 3      /* unblocked, one workgroup per matrix      */
#define BANDLU_GETRF_BLOCKED 4      /* blocked, exact rank-1 trailing updates   */
#define BANDLU_GETRF_BLOCKED_MFMA 5 /* blocked, fp64 MFMA trailing update       */
#define BANDLU_GETRF_SPLIT 6        /* register window + a pivot wavefront      */
#define BANDLU_GETRF_DIAG 7         /* diagonal pivots verified per column, the */
                                    /* split kernel from the first failing one  */
#define BANDLU_GETRF_WIDE 8         /* one persistent launch: blocks of 32      */
                                    /* columns in LDS, matrix-core updates      */
int band_getrf_variant(int64_t n, int64_t kl, int64_t ku, int64_t batch);

/*
 * band_getrf_ex -- band_getrf_batched with the kernel chosen by the caller:
 * variant 0 picks it as band_getrf_batched does, 1..8 forces that
 * BANDLU_GETRF_* kernel.  Arguments 1-10 as in band_getrf_batched (argument
 * 11 is the variant).  A variant that cannot handle the sizes (a window for
 * kl > 31 or a band wider than its registers, a blocked variant for
 * kl > 256) returns BANDLU_ERR_UNSUPPORTED and enqueues nothing.  For tests
 * and measurements that compare the kernels on one input.
 */
int band_getrf_ex(int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab, int64_t strideAB,
                  int32_t *d_ipiv, int64_t strideP, int32_t *d_info, int64_t batch, int variant,
                  void *stream);

/*
 * band_getrs_variant -- which solve kernel band_getrs(_batched) runs for these
 * sizes, with contiguous arguments (ldab = 2kl+ku+1, ldb = n; host-only,
 * enqueues nothing).  Returns one of the BANDLU_GETRS_* codes below, or a
 * negative status for invalid sizes.
 */
#define BANDLU_GETRS_WINDOW 1  /* register window, one wavefront per right-hand side   */
#define BANDLU_GETRS_G16 2     /* register window, 16 lanes per system, many systems    */
#define BANDLU_GETRS_RING 3    /* register ring plus factor columns staged in LDS       */
#define BANDLU_GETRS_GENERIC 4 /* right-hand side in LDS or global memory, any band     */
#define BANDLU_GETRS_LANE 5    /* one lane per row, kl+ku <= 63 and ldab <= 64          */
int band_getrs_variant(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, int64_t batch);

/*
 * band_getrs_ex -- band_getrs_batched with the kernel chosen by the caller:
 * variant 0 picks it as band_getrs_batched does, 1..4 forces that
 * BANDLU_GETRS_* kernel.  Arguments 1-13 as in band_getrs_batched (argument
 * 14 is the variant).  Every variant computes the same sequence of
 * operations, so the results are bitwise equal.  A variant that cannot handle
 * the sizes (a window for kl > 63 or kl+ku >= 128, sixteen lanes for
 * kl+ku > 15, the ring for kl+ku > 1023 or a band of 2 GiB or more) returns
 * BANDLU_ERR_UNSUPPORTED and enqueues nothing.  For tests and measurements
 * that compare the kernels on one input.
 */
int band_getrs_ex(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                  int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                  double *dB, int64_t ldb, int64_t strideB, int64_t batch, int variant,
                  void *stream);

/* Text for a status code (static storage).  The codes follow the LAPACK
 * convention that the paper's callees (xGBTRF, xGETRF; Sec. III-A) use for
 * invalid arguments, plus the two library codes above. */
const char *band_status_string(int status);

/* Details of the last failure on the calling thread ("" if none). */
const char *band_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BANDLU_H */
