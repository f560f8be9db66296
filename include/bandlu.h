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
 *     all buffers passed in are owned and allocated by the caller.  The
 *     library frees none of them and keeps no allocation between calls.  Its
 *     only global state is a thread-local text of the last error and the
 *     fixed per-device array of band_getrf_batched_noalloc.  The one kernel
 *     that needs scratch (band_getrf's persistent wide-band variant) takes it
 *     stream-ordered on the call's stream and returns it the same way.
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
                                    /* (kl <= 7: the pivot decided on scalars)  */
#define BANDLU_GETRF_WINDOW_G16 2   /* register window, 16 lanes per matrix     */
#define BANDLU_GETRF_GENERIC 3      /* unblocked, one workgroup per matrix      */
#define BANDLU_GETRF_BLOCKED 4      /* blocked, exact rank-1 trailing updates   */
#define BANDLU_GETRF_BLOCKED_MFMA 5 /* blocked, fp64 MFMA trailing update       */
#define BANDLU_GETRF_SPLIT 6        /* register window + a pivot wavefront      */
#define BANDLU_GETRF_DIAG 7         /* diagonal pivots verified per column; the */
                                    /* window (kl <= 6) or split kernel from    */
                                    /* the first failing one                    */
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

/*
 * band_gbsv -- steps 3 and 4 in one call (xGBSV): band_getrf on dAB, then
 * band_getrs on the nrhs columns of B (ldb >= n).  dAB, d_ipiv, *d_info and X
 * are those of the two calls, bitwise.  It is band_gbsv_lu followed by
 * band_gbsv_back:
 *   - band_gbsv_lu: band_getrf, and the forward half of the solve,
 *     B <- L^-1 P B.  When the persistent wide-band LU factors the matrix (see
 *     band_getrf) and nrhs <= 33, the forward half runs inside that launch:
 *     one more workgroup trails the chain of panels and applies each
 *     published panel to the right-hand sides.  When nrhs = 1 and the
 *     64-lane window kernel with scalar pivots factors it (1 <= kl <= 6, see
 *     band_getrf_variant), the forward half runs inside that kernel's column
 *     steps.  Otherwise the forward chain runs after the factorisation.
 *   - band_gbsv_back: the backward half, B <- U^-1 B, from the factors.
 * As in band_getrs, B is solved even when *d_info > 0 (a zero pivot then
 * gives IEEE infinities or NaN; LAPACK's xGBSV would skip the solve).
 * Argument errors follow the order of each declaration.
 */
int band_gbsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, double *dAB, int64_t ldab,
              int32_t *d_ipiv, double *dB, int64_t ldb, int32_t *d_info, void *stream);
int band_gbsv_lu(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, double *dAB, int64_t ldab,
                 int32_t *d_ipiv, double *dB, int64_t ldb, int32_t *d_info, void *stream);
int band_gbsv_back(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                   int64_t ldab, double *dB, int64_t ldb, void *stream);

/* ----------------------------------------------------------------------
 * Beyond the LU path: the other branches and structures the paper points to
 * ---------------------------------------------------------------------- */

/*
 * band_detect_convert -- steps 1 and 2 in one read of the dense matrix
 * (Sec. II-A costs I(N) and C(N); Listing 2's detection and conversion).
 * Detection as band_detect with caps kl_cap, ku_cap (both >= 0 here, at most
 * n-1), d_out = {kl, ku, exceeded} (device int64[3]).  While it scans, every
 * element inside the caps' band (-ku_cap <= i-j <= kl_cap) is also stored in
 * dAB, laid out for the caps (ldab >= 2*kl_cap + ku_cap + 1, element (i, j)
 * at row kl_cap + ku_cap + i - j of column j).
 *   - When exceeded = 0, the band of the detected (kl, ku) starts
 *     s = kl_cap + ku_cap - kl - ku rows into dAB.  So dAB + s with the same
 *     ldab holds exactly what dense_to_band(A, kl, ku) writes (rows
 *     0..2kl+ku, bitwise, fill rows and slots outside the matrix +0.0),
 *     ready for band_getrf(n, kl, ku, dAB + s, ldab, ...).  The host learns
 *     s from the one copy of d_out it makes anyway.  The other rows of dAB
 *     hold unspecified values.
 *   - When exceeded = 1, dAB's contents are unspecified (the scan may have
 *     stopped early); convert with dense_to_band after a full detection.
 * Callers size the caps to the memory they can spare for the band: the
 * array has ldab * n doubles whatever the matrix turns out to be.
 */
int band_detect_convert(const double *dA, int64_t n, int64_t lda, int64_t kl_cap,
                        int64_t ku_cap, int64_t *d_out, double *dAB, int64_t ldab, void *stream);

/*
 * band_detect_convert_batched -- band_detect_convert over `batch` matrices
 * (matrix b at dA + b*strideA, its band array at dAB + b*strideAB), with
 * d_out[3*b..3*b+2] per matrix and d_max = {max kl, max ku, any exceeded}.
 * When no cap is exceeded every band array holds, s = kl_cap + ku_cap -
 * max kl - max ku rows in, the band of the batch maximum (kl, ku), as
 * dense_to_band_batched(A, max kl, max ku) writes it.
 */
int band_detect_convert_batched(const double *dA, int64_t n, int64_t lda, int64_t strideA,
                                int64_t batch, int64_t kl_cap, int64_t ku_cap, int64_t *d_out,
                                int64_t *d_max, double *dAB, int64_t ldab, int64_t strideAB,
                                void *stream);

/*
 * band_trsv -- Listing 1's triangular and diagonal branches (Sec. I-C):
 * when detection finds ku = 0 (lower triangular), kl = 0 (upper triangular)
 * or both (diagonal), A X = B is solved by substitution straight from the
 * converted band, with no factorisation.  dAB is the xGBTRF-layout band of
 * dense_to_band (ldab >= 2kl+ku+1, A(i, j) at row kl+ku+i-j); nrhs columns
 * of B (ldb >= n) are overwritten with X.
 *   lower: for j = 0..n-1:  x_j = b_j / A(j,j); b_i = fma(-A(i,j), x_j, b_i), i = j+1..j+kl
 *   upper: for j = n-1..0:  x_j = b_j / A(j,j); b_i = fma(-A(i,j), x_j, b_i), i = j-ku..j-1
 * so X is bitwise that of those loops.  *d_info (int32) = 0, or j+1 for the
 * first exactly-zero diagonal entry; the substitution runs regardless (IEEE
 * infinities or NaN follow).  kl > 0 and ku > 0 together return -3.
 */
int band_trsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB, int64_t ldab,
              double *dB, int64_t ldb, int32_t *d_info, void *stream);

/* band_trsv over `batch` systems: band b at dAB + b*strideAB, right-hand
 * sides at dB + b*strideB (strideB >= ldb*nrhs), info at d_info[b]. */
int band_trsv_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, double *dB, int64_t ldb, int64_t strideB,
                      int32_t *d_info, int64_t batch, void *stream);

/*
 * band_getrs_t -- solve A^T X = B with band_getrf's factors: the general
 * "A \ B" of Listing 1 (Sec. I-C) on the transpose (xGBTRS, trans = 'T').
 * Arguments as band_getrs.  With A = P_0 L_0 P_1 L_1 ... U:
 *   U^T pass, j = 0..n-1:  b_j = fma(-U(i,j), b_i, b_j) for i = j-kv..j-1 ascending; b_j /= U(j,j)
 *   L^T pass, j = n-2..0:  b_j = fma(-l_t, b_{j+t}, b_j) for t = 1..km ascending;
 *                          swap b_j and b_{ipiv[j]-1}
 * X is bitwise that of those loops.  kl is limited to 7999 (the L^T pass
 * keeps a window of kl + 192 entries in 64 KiB of LDS); beyond that the call
 * returns BANDLU_ERR_UNSUPPORTED.
 */
int band_getrs_t(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                 int64_t ldab, const int32_t *d_ipiv, double *dB, int64_t ldb, void *stream);

/* band_getrs_t over `batch` systems, strides as band_getrs_batched. */
int band_getrs_t_batched(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                         int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                         double *dB, int64_t ldb, int64_t strideB, int64_t batch, void *stream);

/*
 * band_getrf_mn -- band LU with partial pivoting of a rectangular m x n band
 * matrix (xGBTRF with m != n; the column steps of Sec. III-A's banded LU).
 * Element (i, j), 0 <= i < m, at dAB[kl+ku+i-j + j*ldab], ldab >= 2kl+ku+1,
 * 0 <= kl <= max(0, m-1), 0 <= ku <= max(0, n-1).  Column j = 0..min(m,n)-1
 * picks its pivot among rows j..min(m-1, j+kl).  ipiv has min(m, n)
 * entries; info and the update extent are as in band_getrf, and the factors
 * are bitwise those of the unblocked algorithm.  m = n gives band_getrf's
 * result.  One workgroup per matrix.
 */
int band_getrf_mn(int64_t m, int64_t n, int64_t kl, int64_t ku, double *dAB, int64_t ldab,
                  int32_t *d_ipiv, int32_t *d_info, void *stream);

/* band_getrf_mn over `batch` matrices (strideAB >= ldab*n, strideP >=
 * min(m, n), batch <= 65535). */
int band_getrf_mn_batched(int64_t m, int64_t n, int64_t kl, int64_t ku, double *dAB,
                          int64_t ldab, int64_t strideAB, int32_t *d_ipiv, int64_t strideP,
                          int32_t *d_info, int64_t batch, void *stream);

/*
 * band_is_symmetric -- the symmetric structure among those the first step of
 * Sec. II-A identifies: *d_flag (device int32) = 1 if A(i,j) == A(j,i) for
 * every 0 < i-j <= kd (IEEE comparison: -0.0 matches +0.0, a NaN matches
 * nothing), else 0.  Reads only the band of the dense column-major matrix
 * (lda >= max(1, n), 0 <= kd <= max(0, n-1)).
 */
int band_is_symmetric(const double *dA, int64_t n, int64_t lda, int64_t kd, int32_t *d_flag,
                      void *stream);

/*
 * band_pbtrf -- band Cholesky A = L L^T of a symmetric positive definite band
 * matrix: the Cholesky case the paper names beside LU (end of Sec. II-B);
 * xPBTRF, lower.  The lower triangle sits in LAPACK's layout, A(i, j),
 * j <= i <= j+kd, at dAB[i - j + j*ldab], ldab >= kd+1.  dense_to_band(A,
 * kd, 0) gives this layout kd rows into its array.  It is overwritten by L.
 *   - Column j: d = A(j,j).  If not d > 0, then *d_info = j+1 and the
 *     factorisation stops; column j and the kd columns after it keep their
 *     updated values, as in the unblocked algorithm.
 *   - Otherwise L(j,j) = sqrt(d), L(i,j) = A(i,j) * (1/L(j,j)), and the
 *     trailing triangle is updated with one fma per entry and step.  L is
 *     bitwise that of the unblocked loops.
 *   - *d_info = 0 on success.
 */
int band_pbtrf(int64_t n, int64_t kd, double *dAB, int64_t ldab, int32_t *d_info, void *stream);

/* band_pbtrf over `batch` matrices (band b at dAB + b*strideAB, info at
 * d_info[b]). */
int band_pbtrf_batched(int64_t n, int64_t kd, double *dAB, int64_t ldab, int64_t strideAB,
                       int32_t *d_info, int64_t batch, void *stream);

/*
 * band_pbtrs -- solve A X = B with band_pbtrf's factor (xPBTRS, lower):
 * L Y = B forward (divide by L(j,j), then update the kd rows below) and
 * L^T X = Y backward (divide, then update the kd rows above with L(j, i)),
 * one fma per entry and step, bitwise those loops.  nrhs columns of B
 * (ldb >= n), in place.
 */
int band_pbtrs(int64_t n, int64_t kd, int64_t nrhs, const double *dAB, int64_t ldab, double *dB,
               int64_t ldb, void *stream);

/* band_pbtrs over `batch` systems (strides as band_getrs_batched). */
int band_pbtrs_batched(int64_t n, int64_t kd, int64_t nrhs, const double *dAB, int64_t ldab,
                       int64_t strideAB, double *dB, int64_t ldb, int64_t strideB, int64_t batch,
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
