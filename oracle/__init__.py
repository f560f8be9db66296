"""CPU oracle for the structure-aware banded LU path (test infrastructure).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never loads it, and it shares no
code with the HIP implementation: the arithmetic lives in ``bandlu_oracle.c``
(plain sequential C, IEEE binary64, explicit fma, no contraction), and this
module only marshals numpy arrays into it.

Matrices follow the column-major convention of the paper's LAPACK callees: a
numpy array ``T`` of shape (n, lda) in C order holds the column-major matrix A
with ``T[j, i] = A[i, j]`` (row j of T is column j of A).  The band array uses
the same convention with shape (n, ldab).

Sections cited: Sec. II-A (three steps, cost functions I, C, F, f), Sec. III-A
(banded LU via xGBTRF, O(N^2) identification and conversion), Listing 2
(detect -> convert -> banded LU).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bandlu_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i64 = ctypes.c_int64
_pd = ctypes.POINTER(ctypes.c_double)
_pi64 = ctypes.POINTER(ctypes.c_int64)
_pi32 = ctypes.POINTER(ctypes.c_int32)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fp contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
            "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("BANDLU_ORACLE_LIB")  # planted-mistake tests only
        if path is None:
            path = _LIB
            if not os.path.exists(path):
                build(force=True)
        L = ctypes.CDLL(path)
        L.oracle_detect.argtypes = [_pd, _i64, _i64, _i64, _i64, _pi64, _pi64]
        L.oracle_dense_to_band.argtypes = [_pd, _i64, _i64, _i64, _i64, _pd, _i64, _pi64]
        L.oracle_gbtrf.argtypes = [_i64, _i64, _i64, _pd, _i64, _pi32, _pi32, _pi64]
        L.oracle_gbtrs.argtypes = [_i64, _i64, _i64, _i64, _pd, _i64, _pi32, _pd, _i64]
        L.oracle_dense_gepp.argtypes = [_i64, _pd, _i64, _pi32, _pi32]
        L.oracle_band_backward_error.argtypes = [_i64, _i64, _i64, _pd, _pd, _i64, _pi32]
        L.oracle_band_trsv.argtypes = [_i64, _i64, _i64, _i64, _pd, _i64, _pd, _i64, _pi32]
        L.oracle_gbtrs_t.argtypes = [_i64, _i64, _i64, _i64, _pd, _i64, _pi32, _pd, _i64]
        L.oracle_gbtrf_mn.argtypes = [_i64, _i64, _i64, _i64, _pd, _i64, _pi32, _pi32, _pi64]
        L.oracle_pbtrf.argtypes = [_i64, _i64, _pd, _i64, _pi32]
        L.oracle_pbtrs.argtypes = [_i64, _i64, _i64, _pd, _i64, _pd, _i64]
        L.oracle_is_symmetric_band.argtypes = [_pd, _i64, _i64, _i64]
        L.oracle_band_backward_error.restype = ctypes.c_double
        for f in ("oracle_detect", "oracle_dense_to_band", "oracle_gbtrf",
                  "oracle_gbtrs", "oracle_dense_gepp"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _dptr(a):
    return a.ctypes.data_as(_pd)


def _check_cm(T, n, name):
    if T.dtype != np.float64 or not T.flags.c_contiguous or T.ndim != 2 or T.shape[0] != n:
        raise ValueError(f"{name}: expected C-contiguous float64 array of shape (n, ld)")


def _status(rc, fn):
    if rc != 0:
        raise ValueError(f"{fn}: invalid argument {-rc}")


def detect(T, kl_cap=-1, ku_cap=-1):
    """Return (kl, ku, exceeded, inspected) for column-major A stored as T[j, i]."""
    n, lda = T.shape
    _check_cm(T, n, "detect")
    out = np.zeros(3, dtype=np.int64)
    cnt = ctypes.c_int64(0)
    rc = lib().oracle_detect(_dptr(T), n, max(lda, 1), kl_cap, ku_cap,
                             out.ctypes.data_as(_pi64), ctypes.byref(cnt))
    _status(rc, "detect")
    return int(out[0]), int(out[1]), int(out[2]), int(cnt.value)


def dense_to_band(T, kl, ku, ldab=None, AB=None):
    """Pack column-major A (T[j, i]) into xGBTRF layout; returns (AB, written).

    AB has shape (n, ldab) with AB[j, r] = band row r of column j.
    """
    n, lda = T.shape
    _check_cm(T, n, "dense_to_band")
    if ldab is None:
        ldab = 2 * kl + ku + 1
    if AB is None:
        AB = np.full((n, ldab), np.nan)  # rows beyond 2kl+ku stay as given
    cnt = ctypes.c_int64(0)
    rc = lib().oracle_dense_to_band(_dptr(T), n, max(lda, 1), kl, ku, _dptr(AB),
                                    ldab, ctypes.byref(cnt))
    _status(rc, "dense_to_band")
    return AB, int(cnt.value)


def gbtrf(AB, kl, ku):
    """Band LU in place on AB (shape (n, ldab)); returns (ipiv int32 1-based, info, flops)."""
    n, ldab = AB.shape
    _check_cm(AB, n, "gbtrf")
    ipiv = np.zeros(max(n, 1), dtype=np.int32)[:n]
    info = ctypes.c_int32(0)
    fl = ctypes.c_int64(0)
    rc = lib().oracle_gbtrf(n, kl, ku, _dptr(AB), ldab, ipiv.ctypes.data_as(_pi32),
                            ctypes.byref(info), ctypes.byref(fl))
    _status(rc, "gbtrf")
    return ipiv, int(info.value), int(fl.value)


def gbtrs(AB, kl, ku, ipiv, B):
    """Solve in place; B has shape (nrhs, ldb) with B[k, i] = rhs k, row i."""
    n, ldab = AB.shape
    _check_cm(AB, n, "gbtrs")
    if B.dtype != np.float64 or not B.flags.c_contiguous or B.ndim != 2:
        raise ValueError("gbtrs: B must be C-contiguous float64 (nrhs, ldb)")
    nrhs, ldb = B.shape
    ipiv = np.ascontiguousarray(ipiv, dtype=np.int32)
    rc = lib().oracle_gbtrs(n, kl, ku, nrhs, _dptr(AB), ldab, ipiv.ctypes.data_as(_pi32),
                            _dptr(B), max(ldb, 1))
    _status(rc, "gbtrs")
    return B


def dense_gepp(T):
    """Dense LU with partial pivoting in place on T (column-major A as T[j, i])."""
    n, lda = T.shape
    _check_cm(T, n, "dense_gepp")
    ipiv = np.zeros(max(n, 1), dtype=np.int32)[:n]
    info = ctypes.c_int32(0)
    rc = lib().oracle_dense_gepp(n, _dptr(T), max(lda, 1), ipiv.ctypes.data_as(_pi32),
                                 ctypes.byref(info))
    _status(rc, "dense_gepp")
    return ipiv, int(info.value)


def band_backward_error(AB0, ABf, kl, ku, ipiv):
    """||A - P L U||_F / (||A||_F n eps) from the band arrays (no dense matrix)."""
    n, ldab = AB0.shape
    _check_cm(AB0, n, "band_backward_error")
    _check_cm(ABf, n, "band_backward_error")
    ipiv = np.ascontiguousarray(ipiv, dtype=np.int32)
    return float(lib().oracle_band_backward_error(n, kl, ku, _dptr(AB0), _dptr(ABf), ldab,
                                                  ipiv.ctypes.data_as(_pi32)))


def op_counts(n, kl, ku):
    """Model operation counts of Sec. II-A for one n x n matrix (reporting only).

    I = n^2 elements inspected, C = (2kl+ku+1) n band slots written,
    f = 2 n kl (kl+ku+1) (the banded LU bound with pivot fill), F = 2/3 n^3.
    """
    I = n * n
    C = (2 * kl + ku + 1) * n
    f = 2 * n * kl * (kl + ku + 1)
    F = 2.0 * n ** 3 / 3.0
    return {"I": I, "C": C, "f": f, "F": F,
            "speedup_ratio": F / (I + C + f) if (I + C + f) else float("inf"),
            "speedup_constraint": (I + C + f) < F,
            "slowdown_constraint": I <= F}


def _rhs(B, fn):
    if B.dtype != np.float64 or not B.flags.c_contiguous or B.ndim != 2:
        raise ValueError(f"{fn}: B must be C-contiguous float64 (nrhs, ldb)")
    return B.shape


def band_trsv(AB, kl, ku, B):
    """Listing 1's triangular / diagonal solve in place on B (nrhs, ldb) from
    the xGBTRF-layout band AB (n, ldab) with kl = 0 or ku = 0; returns info
    (1-based index of the first zero diagonal entry, or 0)."""
    n, ldab = AB.shape
    _check_cm(AB, n, "band_trsv")
    nrhs, ldb = _rhs(B, "band_trsv")
    info = ctypes.c_int32(0)
    rc = lib().oracle_band_trsv(n, kl, ku, nrhs, _dptr(AB), ldab, _dptr(B), max(ldb, 1),
                                ctypes.byref(info))
    _status(rc, "band_trsv")
    return int(info.value)


def gbtrs_t(AB, kl, ku, ipiv, B):
    """Solve A^T x = b in place with the band LU factors; B is (nrhs, ldb)."""
    n, ldab = AB.shape
    _check_cm(AB, n, "gbtrs_t")
    nrhs, ldb = _rhs(B, "gbtrs_t")
    ipiv = np.ascontiguousarray(ipiv, dtype=np.int32)
    rc = lib().oracle_gbtrs_t(n, kl, ku, nrhs, _dptr(AB), ldab, ipiv.ctypes.data_as(_pi32),
                              _dptr(B), max(ldb, 1))
    _status(rc, "gbtrs_t")
    return B


def gbtrf_mn(AB, m, kl, ku):
    """Band LU of an m x n band matrix in place on AB (shape (n, ldab));
    returns (ipiv int32 1-based, length min(m, n), info, flops)."""
    n, ldab = AB.shape
    _check_cm(AB, n, "gbtrf_mn")
    ipiv = np.zeros(max(min(m, n), 1), dtype=np.int32)[:min(m, n)]
    info = ctypes.c_int32(0)
    fl = ctypes.c_int64(0)
    rc = lib().oracle_gbtrf_mn(m, n, kl, ku, _dptr(AB), ldab, ipiv.ctypes.data_as(_pi32),
                               ctypes.byref(info), ctypes.byref(fl))
    _status(rc, "gbtrf_mn")
    return ipiv, int(info.value), int(fl.value)


def dense_to_band_mn(T, m, kl, ku, ldab=None):
    """Pack an m x n column-major matrix (T[j, i] = A[i, j], T of shape (n, >= m))
    into the xGBTRF layout (plain slot loop; every slot outside the matrix or
    the band is +0.0)."""
    n = T.shape[0]
    ldab = 2 * kl + ku + 1 if ldab is None else ldab
    AB = np.zeros((n, ldab))
    for j in range(n):
        for i in range(max(0, j - ku), min(m - 1, j + kl) + 1):
            AB[j, kl + ku + i - j] = T[j, i]
    return AB


def pbtrf(AB, kd):
    """Band Cholesky in place on the lower band AB (shape (n, ldab), element
    (i, j) at AB[j, i - j]); returns info."""
    n, ldab = AB.shape
    _check_cm(AB, n, "pbtrf")
    info = ctypes.c_int32(0)
    rc = lib().oracle_pbtrf(n, kd, _dptr(AB), ldab, ctypes.byref(info))
    _status(rc, "pbtrf")
    return int(info.value)


def pbtrs(AB, kd, B):
    """Solve with the band Cholesky factor in place on B (nrhs, ldb)."""
    n, ldab = AB.shape
    _check_cm(AB, n, "pbtrs")
    nrhs, ldb = _rhs(B, "pbtrs")
    rc = lib().oracle_pbtrs(n, kd, nrhs, _dptr(AB), ldab, _dptr(B), max(ldb, 1))
    _status(rc, "pbtrs")
    return B


def is_symmetric_band(T, kd):
    """1 if A(i, j) == A(j, i) for 0 < i - j <= kd (T[j, i] = A[i, j])."""
    n, lda = T.shape
    _check_cm(T, n, "is_symmetric_band")
    return int(lib().oracle_is_symmetric_band(_dptr(T), n, max(lda, 1), kd))


def lower_band(T, kd, ldab=None):
    """The lower band of a symmetric matrix in LAPACK's lower layout, element
    (i, j), j <= i <= j + kd, at AB[j, i - j]; other slots +0.0."""
    n = T.shape[0]
    ldab = kd + 1 if ldab is None else ldab
    AB = np.zeros((n, ldab))
    for j in range(n):
        for i in range(j, min(n - 1, j + kd) + 1):
            AB[j, i - j] = T[j, i]
    return AB


def detect_convert(T, kl_cap, ku_cap):
    """The fused identify-and-convert pass as its definition: detection with
    the caps, and when no cap is exceeded the band of the detected (kl, ku)
    in the xGBTRF layout.  Returns (kl, ku, exceeded, AB or None)."""
    kl, ku, ex, _ = detect(T, kl_cap, ku_cap)
    if ex:
        return kl, ku, ex, None
    AB, _ = dense_to_band(T, kl, ku)
    return kl, ku, ex, AB
