/*
 * CPU oracle for the structure-aware banded LU path
 * ("When Structure is Silent", Sec. II-A three-step strategy, Sec. III,
 * Listing 2: detect -> convert to band format -> banded LU).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file.  It may be used by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, and by nothing else.  It shares no code, no
 * header and no constant with the HIP implementation.
 *
 * Everything is plain, slow, sequential C in IEEE binary64.  Build with
 * -ffp-contract=off: every fused multiply-add below is an explicit fma() and no
 * other expression may be contracted.
 *
 * Conventions (the paper names the routines, LAPACK fixes their contracts):
 *   - dense A is column-major, element (i, j) at A[i + j*lda], 0-based;
 *   - the band array AB follows the LAPACK xGBTRF layout: matrix element
 *     (i, j) lives at AB[kl + ku + i - j + j*ldab], ldab >= 2*kl + ku + 1; rows
 *     0..kl-1 of AB hold the fill-in that partial pivoting creates in U;
 *   - ipiv is 1-based int32 as in xGBTRF; info = 0 or the 1-based index of
 *     the first exactly-zero pivot.
 *
 * Return values: 0 on success, -k if argument k (1-based) is invalid.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static int64_t imin(int64_t a, int64_t b) { return a < b ? a : b; }
static int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }

/* ---------------------------------------------------------------------------
 * Step 1, identify the structure: I(N) of Sec. II-A, an O(N^2) element scan
 * (Sec. III-A, Eq. for I(N), C(N)).  The paper gives no body for its
 * banded-structure predicate; the reading taken here returns the exact lower
 * and upper bandwidths over the entries that compare unequal to 0.0 (so -0.0
 * counts as zero and NaN as nonzero).  Caps < 0 mean "no cap"; out[2] reports
 * whether a bandwidth exceeds its cap.
 *
 * out[0] = kl = max(0, max over nonzeros of i - j)
 * out[1] = ku = max(0, max over nonzeros of j - i)
 * out[2] = exceeded flag
 * *inspected = number of elements read (the I(N) operation count).
 * ------------------------------------------------------------------------- */
int oracle_detect(const double *A, int64_t n, int64_t lda, int64_t kl_cap,
                  int64_t ku_cap, int64_t *out, int64_t *inspected)
{
    if (n < 0) return -2;
    if (lda < imax(1, n)) return -3;
    if (!out) return -6;
    int64_t kl = 0, ku = 0, count = 0;
    for (int64_t j = 0; j < n; ++j) {
        for (int64_t i = 0; i < n; ++i) {
            double a = A[i + j * lda];
            ++count;
            if (a != 0.0) {
                if (i - j > kl) kl = i - j;
                if (j - i > ku) ku = j - i;
            }
        }
    }
    out[0] = kl;
    out[1] = ku;
    out[2] = ((kl_cap >= 0 && kl > kl_cap) || (ku_cap >= 0 && ku > ku_cap)) ? 1 : 0;
    if (inspected) *inspected = count;
    return 0;
}

/* ---------------------------------------------------------------------------
 * Step 2, convert: C(N) of Sec. II-A, the dense -> band copy that Listing 2
 * performs before calling the banded LU.  The target is the xGBTRF layout.
 * Every slot of rows 0..2kl+ku of AB is written exactly once: in-band matrix
 * entries are copied bit for bit (so -0.0 and NaN payloads survive), every
 * other slot (fill rows, corners outside the matrix) becomes +0.0.  Rows
 * >= 2kl+ku+1 (when ldab is larger) are not touched.  Entries of A outside
 * the given (kl, ku) are dropped.
 * *written = number of AB slots written (the C(N) operation count).
 * ------------------------------------------------------------------------- */
int oracle_dense_to_band(const double *A, int64_t n, int64_t lda, int64_t kl,
                         int64_t ku, double *AB, int64_t ldab, int64_t *written)
{
    if (n < 0) return -2;
    if (lda < imax(1, n)) return -3;
    if (kl < 0 || kl > imax(0, n - 1)) return -4;
    if (ku < 0 || ku > imax(0, n - 1)) return -5;
    if (ldab < 2 * kl + ku + 1) return -7;
    int64_t rows = 2 * kl + ku + 1, count = 0;
    for (int64_t j = 0; j < n; ++j) {
        for (int64_t r = 0; r < rows; ++r) {
            int64_t i = r - kl - ku + j; /* matrix row of this slot */
            double *dst = &AB[r + j * ldab];
            if (r >= kl && i >= 0 && i < n) {
                memcpy(dst, &A[i + j * lda], sizeof(double));
            } else {
                uint64_t zero = 0;
                memcpy(dst, &zero, sizeof(double));
            }
            ++count;
        }
    }
    if (written) *written = count;
    return 0;
}

/* ---------------------------------------------------------------------------
 * Step 3, specialised algorithm: f(N) of Sec. II-A / Sec. III-A, the banded LU
 * with partial pivoting that the paper dispatches to (xGBTRF), unblocked,
 * one column at a time.  With kv = kl + ku:
 *
 *   zero every in-matrix fill slot (AB rows 0..kl-1 whose matrix row is >= 0);
 *   ju = 0
 *   for j = 0 .. n-1:
 *     km = min(kl, n-1-j)
 *     p  = first index t in 0..km with the largest |a(j+t, j)|, taking a new
 *          candidate only when strictly larger (BLAS i_amax convention)
 *     ipiv[j] = j + p + 1
 *     if a(j+p, j) != 0:
 *        ju = max(ju, min(j + ku + p, n-1))
 *        swap rows j and j+p over columns j..ju
 *        if |pivot| >= DBL_MIN: r = 1/pivot, l_t = a(j+t, j) * r
 *        else:                   l_t = a(j+t, j) / pivot
 *        for c = j+1..ju, t = 1..km:  a(j+t, c) = fma(-l_t, a(j, c), a(j+t, c))
 *     else if info == 0: info = j + 1
 *
 * The multipliers of column j are stored where they are computed and are not
 * permuted by later interchanges (product form of L, as xGBTRF).
 * *flops = number of floating-point operations executed (2 per fma, 1 per
 * scaling), the f(N) operation count.
 * ------------------------------------------------------------------------- */
int oracle_gbtrf(int64_t n, int64_t kl, int64_t ku, double *AB, int64_t ldab,
                 int32_t *ipiv, int32_t *info, int64_t *flops)
{
    if (n < 0) return -1;
    if (kl < 0 || kl > imax(0, n - 1)) return -2;
    if (ku < 0 || ku > imax(0, n - 1)) return -3;
    if (ldab < 2 * kl + ku + 1) return -5;
    const int64_t kv = kl + ku;
    int64_t count = 0;
    *info = 0;
#define AT(i, c) AB[kv + (i) - (c) + (c) * ldab]
    /* fill-in slots inside the matrix start at zero */
    for (int64_t c = 0; c < n; ++c)
        for (int64_t r = imax(0, kv - c); r < kl; ++r) AB[r + c * ldab] = 0.0;

    int64_t ju = 0;
    for (int64_t j = 0; j < n; ++j) {
        int64_t km = imin(kl, n - 1 - j);
        int64_t p = 0;
        double dmax = fabs(AT(j, j));
        for (int64_t t = 1; t <= km; ++t) {
            if (fabs(AT(j + t, j)) > dmax) {
                p = t;
                dmax = fabs(AT(j + t, j));
            }
        }
        ipiv[j] = (int32_t)(j + p + 1);
        if (AT(j + p, j) != 0.0) {
            ju = imax(ju, imin(j + ku + p, n - 1));
            if (p != 0) {
                for (int64_t c = j; c <= ju; ++c) {
                    double tmp = AT(j, c);
                    AT(j, c) = AT(j + p, c);
                    AT(j + p, c) = tmp;
                }
            }
            if (km > 0) {
                double piv = AT(j, j);
                if (fabs(piv) >= DBL_MIN) {
                    double r = 1.0 / piv;
                    for (int64_t t = 1; t <= km; ++t) AT(j + t, j) = AT(j + t, j) * r;
                } else {
                    for (int64_t t = 1; t <= km; ++t) AT(j + t, j) = AT(j + t, j) / piv;
                }
                count += km;
                for (int64_t c = j + 1; c <= ju; ++c) {
                    double u = AT(j, c);
                    for (int64_t t = 1; t <= km; ++t)
                        AT(j + t, c) = fma(-AT(j + t, j), u, AT(j + t, c));
                }
                count += 2 * km * (ju - j);
            }
        } else if (*info == 0) {
            *info = (int32_t)(j + 1);
        }
    }
#undef AT
    if (flops) *flops = count;
    return 0;
}

/* ---------------------------------------------------------------------------
 * Solve with the factors (the "lu(A) \ B" of Listing 1 / Listing 2, i.e.
 * xGBTRS with no transpose), nrhs right-hand sides in column-major B.
 *   forward:  for j = 0..n-2: swap b[j], b[ipiv[j]-1];
 *                             b[j+t] = fma(-l_t, b[j], b[j+t]), t = 1..km
 *   backward: for j = n-1..0: b[j] = b[j] / U(j,j);
 *                             b[i] = fma(-U(i,j), b[j], b[i]), i = max(0,j-kv)..j-1
 * ------------------------------------------------------------------------- */
int oracle_gbtrs(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *AB,
                 int64_t ldab, const int32_t *ipiv, double *B, int64_t ldb)
{
    if (n < 0) return -1;
    if (kl < 0 || kl > imax(0, n - 1)) return -2;
    if (ku < 0 || ku > imax(0, n - 1)) return -3;
    if (nrhs < 0) return -4;
    if (ldab < 2 * kl + ku + 1) return -6;
    if (ldb < imax(1, n)) return -9;
    const int64_t kv = kl + ku;
#define AT(i, c) AB[kv + (i) - (c) + (c) * ldab]
    for (int64_t k = 0; k < nrhs; ++k) {
        double *b = B + k * ldb;
        if (kl > 0) {
            for (int64_t j = 0; j < n - 1; ++j) {
                int64_t km = imin(kl, n - 1 - j);
                int64_t l = ipiv[j] - 1;
                if (l != j) {
                    double tmp = b[l];
                    b[l] = b[j];
                    b[j] = tmp;
                }
                for (int64_t t = 1; t <= km; ++t) b[j + t] = fma(-AT(j + t, j), b[j], b[j + t]);
            }
        }
        for (int64_t j = n - 1; j >= 0; --j) {
            b[j] = b[j] / AT(j, j);
            for (int64_t i = imax(0, j - kv); i < j; ++i) b[i] = fma(-AT(i, j), b[j], b[i]);
        }
    }
#undef AT
    return 0;
}

/* ---------------------------------------------------------------------------
 * Brute force for pinning oracle_gbtrf: plain dense Gaussian elimination with
 * partial pivoting (the generic xGETRF-class algorithm of Sec. III-A, F(N)),
 * written independently of the band code.  Whole rows are interchanged
 * (LAPACK xGETF2 convention), so L comes out in its final permuted form.  The
 * same arithmetic rules as the band routine are used (reciprocal scaling when
 * |pivot| >= DBL_MIN, one fma per update), so on a banded input the pivots
 * and U agree exactly with the band routine.
 * ------------------------------------------------------------------------- */
int oracle_dense_gepp(int64_t n, double *A, int64_t lda, int32_t *ipiv, int32_t *info)
{
    if (n < 0) return -1;
    if (lda < imax(1, n)) return -3;
    *info = 0;
    for (int64_t k = 0; k < n; ++k) {
        int64_t p = k;
        double best = fabs(A[k + k * lda]);
        for (int64_t i = k + 1; i < n; ++i) {
            double v = fabs(A[i + k * lda]);
            if (v > best) {
                best = v;
                p = i;
            }
        }
        ipiv[k] = (int32_t)(p + 1);
        if (A[p + k * lda] == 0.0) {
            if (*info == 0) *info = (int32_t)(k + 1);
            continue;
        }
        if (p != k) {
            for (int64_t c = 0; c < n; ++c) {
                double tmp = A[k + c * lda];
                A[k + c * lda] = A[p + c * lda];
                A[p + c * lda] = tmp;
            }
        }
        double piv = A[k + k * lda];
        if (fabs(piv) >= DBL_MIN) {
            double r = 1.0 / piv;
            for (int64_t i = k + 1; i < n; ++i) A[i + k * lda] *= r;
        } else {
            for (int64_t i = k + 1; i < n; ++i) A[i + k * lda] /= piv;
        }
        for (int64_t c = k + 1; c < n; ++c)
            for (int64_t i = k + 1; i < n; ++i)
                A[i + c * lda] = fma(-A[i + k * lda], A[k + c * lda], A[i + c * lda]);
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Backward error of a band factorization, without forming anything dense:
 *   rebuild M = P_0 L_0 P_1 L_1 ... P_{n-1} L_{n-1} U from the factors in band
 *   storage (lower bandwidth kl, upper kv), in long double, and return
 *   ||A - M||_F / (||A||_F * n * eps)  with A given as the unfactored band
 *   array AB0 (the output of the conversion step).
 * Returns a negative value if the reconstruction needs an entry outside the
 * band (which would mean the factors violate the fill bound of xGBTRF).
 * ------------------------------------------------------------------------- */
double oracle_band_backward_error(int64_t n, int64_t kl, int64_t ku, const double *AB0,
                                  const double *ABf, int64_t ldab, const int32_t *ipiv)
{
    const int64_t kv = kl + ku;
    const int64_t lw = kl + kv + 1; /* rows of the work band: kv above, kl below */
    if (n == 0) return 0.0;
    long double *M = (long double *)calloc((size_t)(lw * n), sizeof(long double));
    if (!M) return -2.0;
    /* M(i, c) at M[kv + i - c + c*lw], valid for c-kv <= i <= c+kl */
#define MAT(i, c) M[kv + (i) - (c) + (c) * lw]
#define FAT(i, c) ABf[kv + (i) - (c) + (c) * ldab]
    for (int64_t c = 0; c < n; ++c)
        for (int64_t i = imax(0, c - kv); i <= c; ++i) MAT(i, c) = FAT(i, c);
    for (int64_t j = n - 1; j >= 0; --j) {
        int64_t km = imin(kl, n - 1 - j);
        int64_t cend = imin(n - 1, j + kv);
        /* M <- L_j M : row_{j+t} += l_t * row_j */
        for (int64_t t = 1; t <= km; ++t) {
            long double l = FAT(j + t, j);
            for (int64_t c = j; c <= cend; ++c) {
                long double v = MAT(j, c);
                if (v == 0.0L) continue;
                int64_t i = j + t;
                if (i - c > kl || c - i > kv) { free(M); return -1.0; }
                MAT(i, c) += l * v;
            }
        }
        /* M <- P_j M : swap rows j and q over the columns where either is stored */
        int64_t q = ipiv[j] - 1;
        if (q != j) {
            int64_t c0 = imax(0, q - kl), c1 = imin(n - 1, j + kv);
            for (int64_t c = c0; c <= c1; ++c) {
                int inj = (j - c <= kl) && (c - j <= kv);
                int inq = (q - c <= kl) && (c - q <= kv);
                long double vj = inj ? MAT(j, c) : 0.0L;
                long double vq = inq ? MAT(q, c) : 0.0L;
                if ((!inj && vq != 0.0L) || (!inq && vj != 0.0L)) { free(M); return -1.0; }
                if (inj) MAT(j, c) = vq;
                if (inq) MAT(q, c) = vj;
            }
        }
    }
    long double num = 0.0L, den = 0.0L;
    for (int64_t c = 0; c < n; ++c) {
        for (int64_t i = imax(0, c - kv); i <= imin(n - 1, c + kl); ++i) {
            long double a = 0.0L;
            if (c - i <= ku) a = AB0[kv + i - c + c * ldab];
            long double d = a - MAT(i, c);
            num += d * d;
            den += a * a;
        }
    }
#undef MAT
#undef FAT
    free(M);
    if (den == 0.0L) return num == 0.0L ? 0.0 : INFINITY;
    return (double)(sqrtl(num) / (sqrtl(den) * (long double)n * (long double)DBL_EPSILON));
}

/* ---------------------------------------------------------------------------
 * Listing 1's triangular and diagonal branches (Sec. I-C): when the detected
 * band has ku = 0 (lower triangular), kl = 0 (upper triangular) or both
 * (diagonal), A x = b is solved by substitution straight from the band array,
 * with no factorisation.  AB is in the xGBTRF layout of the conversion step
 * (element (i, j) at AB[kl + ku + i - j + j*ldab]), nrhs right-hand sides in
 * column-major B, solved in place.
 *
 *   lower (ku = 0):  for j = 0..n-1:   b[j] = b[j] / A(j,j);
 *                                      b[i] = fma(-A(i,j), b[j], b[i]), i = j+1..min(n-1, j+kl)
 *   upper (kl = 0):  for j = n-1..0:   b[j] = b[j] / A(j,j);
 *                                      b[i] = fma(-A(i,j), b[j], b[i]), i = max(0, j-ku)..j-1
 *   (kl = ku = 0 is both: b[j] = b[j] / A(j,j).)
 *
 * *info = 0, or j+1 for the first exactly-zero diagonal entry A(j,j); the
 * substitution runs regardless (a zero divisor gives IEEE infinities or NaN).
 * Returns -3 if the band is not triangular (kl > 0 and ku > 0).
 * ------------------------------------------------------------------------- */
int oracle_band_trsv(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *AB,
                     int64_t ldab, double *B, int64_t ldb, int32_t *info)
{
    if (n < 0) return -1;
    if (kl < 0 || kl > imax(0, n - 1)) return -2;
    if (ku < 0 || ku > imax(0, n - 1)) return -3;
    if (kl > 0 && ku > 0) return -3;
    if (nrhs < 0) return -4;
    if (ldab < 2 * kl + ku + 1) return -6;
    if (ldb < imax(1, n)) return -8;
    const int64_t kv = kl + ku;
#define AT(i, c) AB[kv + (i) - (c) + (c) * ldab]
    *info = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (AT(j, j) == 0.0) {
            *info = (int32_t)(j + 1);
            break;
        }
    }
    for (int64_t k = 0; k < nrhs; ++k) {
        double *b = B + k * ldb;
        if (ku == 0) {
            for (int64_t j = 0; j < n; ++j) {
                b[j] = b[j] / AT(j, j);
                for (int64_t i = j + 1; i <= imin(n - 1, j + kl); ++i)
                    b[i] = fma(-AT(i, j), b[j], b[i]);
            }
        } else {
            for (int64_t j = n - 1; j >= 0; --j) {
                b[j] = b[j] / AT(j, j);
                for (int64_t i = imax(0, j - ku); i < j; ++i) b[i] = fma(-AT(i, j), b[j], b[i]);
            }
        }
    }
#undef AT
    return 0;
}

/* ---------------------------------------------------------------------------
 * Solve with the transpose, A^T x = b, from the band LU factors (the general
 * "A \ B" of Listing 1 applied to A^T; xGBTRS with trans = 'T').  With
 * A = P_0 L_0 P_1 L_1 ... U (product form), A^T = U^T ... L_1^T P_1 L_0^T P_0:
 *
 *   U^T pass, forward:  for j = 0..n-1:
 *       b[j] = fma(-U(i,j), b[i], b[j]) for i = max(0, j-kv)..j-1 (ascending);
 *       b[j] = b[j] / U(j,j)
 *   L^T pass, backward (kl > 0):  for j = n-2..0, km = min(kl, n-1-j):
 *       b[j] = fma(-l_t, b[j+t], b[j]) for t = 1..km (ascending), l_t = AB row kv+t of column j;
 *       swap b[j] and b[ipiv[j]-1]
 * ------------------------------------------------------------------------- */
int oracle_gbtrs_t(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *AB,
                   int64_t ldab, const int32_t *ipiv, double *B, int64_t ldb)
{
    if (n < 0) return -1;
    if (kl < 0 || kl > imax(0, n - 1)) return -2;
    if (ku < 0 || ku > imax(0, n - 1)) return -3;
    if (nrhs < 0) return -4;
    if (ldab < 2 * kl + ku + 1) return -6;
    if (ldb < imax(1, n)) return -9;
    const int64_t kv = kl + ku;
#define AT(i, c) AB[kv + (i) - (c) + (c) * ldab]
    for (int64_t k = 0; k < nrhs; ++k) {
        double *b = B + k * ldb;
        for (int64_t j = 0; j < n; ++j) {
            for (int64_t i = imax(0, j - kv); i < j; ++i) b[j] = fma(-AT(i, j), b[i], b[j]);
            b[j] = b[j] / AT(j, j);
        }
        if (kl > 0) {
            for (int64_t j = n - 2; j >= 0; --j) {
                int64_t km = imin(kl, n - 1 - j);
                for (int64_t t = 1; t <= km; ++t) b[j] = fma(-AT(j + t, j), b[j + t], b[j]);
                int64_t l = ipiv[j] - 1;
                if (l != j) {
                    const double bl = b[l];
                    b[l] = b[j];
                    b[j] = bl;
                }
            }
        }
    }
#undef AT
    return 0;
}

/* ---------------------------------------------------------------------------
 * Band LU with partial pivoting of a rectangular m x n band matrix (xGBTRF
 * with m != n; the same column steps as oracle_gbtrf, Sec. III-A), for
 * j = 0..min(m,n)-1 with km = min(kl, m-1-j) candidates below the diagonal
 * and the update extent ju = max(ju, min(j + ku + p, n-1)).  Element (i, j),
 * 0 <= i < m, lives at AB[kl + ku + i - j + j*ldab]; ipiv has min(m, n)
 * entries.  Fill slots inside the matrix (AB rows 0..kl-1 whose matrix row
 * is >= 0) start at zero.
 * ------------------------------------------------------------------------- */
int oracle_gbtrf_mn(int64_t m, int64_t n, int64_t kl, int64_t ku, double *AB, int64_t ldab,
                    int32_t *ipiv, int32_t *info, int64_t *flops)
{
    if (m < 0) return -1;
    if (n < 0) return -2;
    if (kl < 0 || kl > imax(0, m - 1)) return -3;
    if (ku < 0 || ku > imax(0, n - 1)) return -4;
    if (ldab < 2 * kl + ku + 1) return -6;
    const int64_t kv = kl + ku;
    int64_t count = 0;
    *info = 0;
#define AT(i, c) AB[kv + (i) - (c) + (c) * ldab]
    for (int64_t c = 0; c < n; ++c)
        for (int64_t r = imax(0, kv - c); r < kl; ++r)
            if (r - kv + c < m) AB[r + c * ldab] = 0.0;
    int64_t ju = 0;
    const int64_t steps = imin(m, n);
    for (int64_t j = 0; j < steps; ++j) {
        const int64_t km = imin(kl, m - 1 - j);
        int64_t p = 0;
        double best = fabs(AT(j, j));
        for (int64_t t = 1; t <= km; ++t) {
            const double v = fabs(AT(j + t, j));
            if (v > best) {
                best = v;
                p = t;
            }
        }
        ipiv[j] = (int32_t)(j + p + 1);
        if (AT(j + p, j) == 0.0) {
            if (*info == 0) *info = (int32_t)(j + 1);
            continue;
        }
        ju = imax(ju, imin(n - 1, j + ku + p));
        for (int64_t c = j; p != 0 && c <= ju; ++c) {
            const double t0 = AT(j, c);
            AT(j, c) = AT(j + p, c);
            AT(j + p, c) = t0;
        }
        if (km == 0) continue;
        const double piv = AT(j, j);
        if (fabs(piv) >= DBL_MIN) {
            const double r = 1.0 / piv;
            for (int64_t t = 1; t <= km; ++t) AT(j + t, j) *= r;
        } else {
            for (int64_t t = 1; t <= km; ++t) AT(j + t, j) /= piv;
        }
        count += km;
        for (int64_t c = j + 1; c <= ju; ++c)
            for (int64_t t = 1; t <= km; ++t)
                AT(j + t, c) = fma(-AT(j + t, j), AT(j, c), AT(j + t, c));
        count += 2 * km * (ju - j);
    }
#undef AT
    if (flops) *flops = count;
    return 0;
}

/* ---------------------------------------------------------------------------
 * Band Cholesky, A = L L^T, for a symmetric positive definite band matrix
 * with kd sub-diagonals (the Cholesky case the paper names beside LU, end of
 * Sec. II-B, on the symmetric structure of Sec. II-A; xPBTRF, lower).  The
 * lower triangle is stored as in LAPACK: element (i, j), j <= i <= j+kd, at
 * AB[i - j + j*ldab], ldab >= kd+1.  Right-looking, column by column:
 *
 *   for j = 0..n-1, kn = min(kd, n-1-j):
 *     d = A(j,j); if not (d > 0): info = j+1, stop (A(j,j) keeps d)
 *     d = sqrt(d); A(j,j) = d; r = 1/d; L(i,j) = A(i,j) * r, i = j+1..j+kn
 *     A(i,c) = fma(-L(i,j), L(c,j), A(i,c)) for c = j+1..j+kn, i = c..j+kn
 * ------------------------------------------------------------------------- */
int oracle_pbtrf(int64_t n, int64_t kd, double *AB, int64_t ldab, int32_t *info)
{
    if (n < 0) return -1;
    if (kd < 0 || kd > imax(0, n - 1)) return -2;
    if (ldab < kd + 1) return -4;
#define LT(i, c) AB[(i) - (c) + (c) * ldab]
    *info = 0;
    for (int64_t j = 0; j < n; ++j) {
        const int64_t kn = imin(kd, n - 1 - j);
        const double d0 = LT(j, j);
        if (!(d0 > 0.0)) {
            *info = (int32_t)(j + 1);
            break;
        }
        const double d = sqrt(d0);
        LT(j, j) = d;
        const double r = 1.0 / d;
        for (int64_t i = j + 1; i <= j + kn; ++i) LT(i, j) = LT(i, j) * r;
        for (int64_t c = j + 1; c <= j + kn; ++c)
            for (int64_t i = c; i <= j + kn; ++i) LT(i, c) = fma(-LT(i, j), LT(c, j), LT(i, c));
    }
#undef LT
    return 0;
}

/* ---------------------------------------------------------------------------
 * Solve A x = b with the band Cholesky factor (xPBTRS, lower):
 *   L y = b,   forward:  for j = 0..n-1:  b[j] = b[j] / L(j,j);
 *                                         b[i] = fma(-L(i,j), b[j], b[i]), i = j+1..min(n-1, j+kd)
 *   L^T x = y, backward: for j = n-1..0:  b[j] = b[j] / L(j,j);
 *                                         b[i] = fma(-L(j,i), b[j], b[i]), i = max(0, j-kd)..j-1
 * ------------------------------------------------------------------------- */
int oracle_pbtrs(int64_t n, int64_t kd, int64_t nrhs, const double *AB, int64_t ldab, double *B,
                 int64_t ldb)
{
    if (n < 0) return -1;
    if (kd < 0 || kd > imax(0, n - 1)) return -2;
    if (nrhs < 0) return -3;
    if (ldab < kd + 1) return -5;
    if (ldb < imax(1, n)) return -7;
#define LT(i, c) AB[(i) - (c) + (c) * ldab]
    for (int64_t k = 0; k < nrhs; ++k) {
        double *b = B + k * ldb;
        for (int64_t j = 0; j < n; ++j) {
            b[j] = b[j] / LT(j, j);
            for (int64_t i = j + 1; i <= imin(n - 1, j + kd); ++i) b[i] = fma(-LT(i, j), b[j], b[i]);
        }
        for (int64_t j = n - 1; j >= 0; --j) {
            b[j] = b[j] / LT(j, j);
            for (int64_t i = imax(0, j - kd); i < j; ++i) b[i] = fma(-LT(j, i), b[j], b[i]);
        }
    }
#undef LT
    return 0;
}

/* ---------------------------------------------------------------------------
 * Symmetry of a band (the symmetric structure of Sec. II-A's first step,
 * examined as Listing 1's text describes): 1 if A(i,j) == A(j,i) under IEEE
 * comparison for every 0 < i-j <= kd (so -0.0 matches +0.0 and a NaN matches
 * nothing), else 0.  Entries beyond kd are not examined (the detected
 * bandwidths already say they are zero).
 * ------------------------------------------------------------------------- */
int oracle_is_symmetric_band(const double *A, int64_t n, int64_t lda, int64_t kd)
{
    for (int64_t j = 0; j < n; ++j)
        for (int64_t i = j + 1; i <= imin(n - 1, j + kd); ++i)
            if (!(A[i + j * lda] == A[j + i * lda])) return 0;
    return 1;
}
