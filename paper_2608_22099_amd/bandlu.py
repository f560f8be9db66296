"""Thin Python binding of libbandlu.so (the C ABI in include/bandlu.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Tensors must be float64 (int32 for pivots) CUDA/ROCm tensors,
C-contiguous in their last dimension, on the current device; work is enqueued
on torch's current stream.  If the library is missing this module raises on
import -- there is no fallback.

Storage convention: a torch tensor ``T`` of shape (n, ld) holds the
column-major matrix A with ``T[j, i] = A[i, j]`` (row j of T is column j of A,
ld >= n is the leading dimension).  Band arrays use the same convention with
shape (n, ldab); batched arrays add a leading batch dimension.

Names follow the paper's path (Sec. II-A, Listing 2): band_detect (identify),
dense_to_band (convert), band_getrf / band_getrf_batched (specialised LU),
band_getrs / band_getrs_batched (solve).  The host policy of Listing 2 (the
Sec. II-B speedup constraint and structure_aware_lu) is in ``policy``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbandlu.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -m paper_2608_22099_amd.build` "
        "(there is no fallback implementation)")

_lib = ctypes.CDLL(LIB_PATH)

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p

EXPORTS = {
    "band_detect": [_vp, _i64, _i64, _i64, _i64, _vp, _vp],
    "band_detect_batched": [_vp, _i64, _i64, _i64, _i64, _i64, _i64, _vp, _vp, _vp],
    "dense_to_band": [_vp, _i64, _i64, _i64, _i64, _vp, _i64, _vp],
    "dense_to_band_batched": [_vp, _i64, _i64, _i64, _i64, _i64, _vp, _i64, _i64, _i64, _vp],
    "band_getrf": [_i64, _i64, _i64, _vp, _i64, _vp, _vp, _vp],
    "band_getrf_batched": [_i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _vp],
    "band_getrf_batched_noalloc": [_i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _vp],
    "band_getrs": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp],
    "band_getrs_batched": [_i64, _i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _i64,
                           _i64, _vp],
    "band_getrf_variant": [_i64, _i64, _i64, _i64],
    "band_getrf_ex": [_i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, ctypes.c_int, _vp],
    "band_getrs_variant": [_i64, _i64, _i64, _i64, _i64],
    "band_getrs_ex": [_i64, _i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _i64, _i64,
                      ctypes.c_int, _vp],
    "band_detect_convert": [_vp, _i64, _i64, _i64, _i64, _vp, _vp, _i64, _vp],
    "band_detect_convert_batched": [_vp, _i64, _i64, _i64, _i64, _i64, _i64, _vp, _vp, _vp, _i64,
                                    _i64, _vp],
    "band_trsv": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp],
    "band_trsv_batched": [_i64, _i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _i64, _vp, _i64,
                          _vp],
    "band_getrs_t": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp],
    "band_getrs_t_batched": [_i64, _i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _i64,
                             _i64, _vp],
    "band_getrf_mn": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _vp],
    "band_getrf_mn_batched": [_i64, _i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _vp],
    "band_is_symmetric": [_vp, _i64, _i64, _i64, _vp, _vp],
    "band_pbtrf": [_i64, _i64, _vp, _i64, _vp, _vp],
    "band_pbtrf_batched": [_i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp],
    "band_pbtrs": [_i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp],
    "band_pbtrs_batched": [_i64, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _i64, _i64, _vp],
    "band_gbsv": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp, _vp],
    "band_gbsv_lu": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp, _vp],
    "band_gbsv_back": [_i64, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp],
    "band_status_string": [ctypes.c_int],
    "band_last_error": [],
}
for _name, _args in EXPORTS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_char_p if _name in ("band_status_string", "band_last_error") \
        else ctypes.c_int

VARIANTS = {1: "window", 2: "window_g16", 3: "generic", 4: "blocked", 5: "blocked_mfma",
            6: "split", 7: "diag", 8: "wide"}
_VARIANT_CODES = {name: code for code, name in VARIANTS.items()}
GETRS_VARIANTS = {1: "window", 2: "g16", 3: "ring", 4: "generic", 5: "lane"}
_GETRS_CODES = {name: code for code, name in GETRS_VARIANTS.items()}


class BandLUError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = _lib.band_last_error().decode() or _lib.band_status_string(status).decode()
        super().__init__(f"{fn} failed with status {status}: {msg}")


def _call(name, *args):
    rc = getattr(_lib, name)(*args)
    if rc != 0:
        raise BandLUError(name, rc)
    return rc


def _stream():
    return _vp(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return _vp(t.data_ptr()) if t is not None and t.numel() else _vp(0)


def _check(t, dtype, name, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a GPU tensor")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name}: expected {ndim} dims, got {t.dim()}")
    if t.numel() and t.stride(-1) != 1:
        raise ValueError(f"{name}: last dimension must be contiguous")


def _ld(t):
    """Leading dimension of a (.., n, ld) tensor whose rows are the columns of A."""
    return max(1, t.stride(-2)) if t.dim() >= 2 and t.shape[-2] > 1 else max(1, t.shape[-1])


# ------------------------------------------------------------------ detect --
def band_detect(A, kl_cap=-1, ku_cap=-1, out=None):
    """(kl, ku, exceeded) of A as a device int64 tensor of 3 (no host sync)."""
    _check(A, torch.float64, "A", 2)
    n = A.shape[0]
    if out is None:
        out = torch.empty(3, dtype=torch.int64, device=A.device)
    _call("band_detect", _ptr(A), n, max(_ld(A), n, 1), kl_cap, ku_cap, _ptr(out), _stream())
    return out


def band_detect_batched(A, kl_cap=-1, ku_cap=-1, out=None, dmax=None):
    """Per-matrix (batch, 3) and batch-max (3,) device int64 tensors."""
    _check(A, torch.float64, "A", 3)
    batch, n = A.shape[0], A.shape[1]
    if out is None:
        out = torch.empty((batch, 3), dtype=torch.int64, device=A.device)
    if dmax is None:
        dmax = torch.empty(3, dtype=torch.int64, device=A.device)
    stride = A.stride(0) if batch > 1 else max(_ld(A), n, 1) * n
    _call("band_detect_batched", _ptr(A), n, max(_ld(A), n, 1), stride, batch, kl_cap, ku_cap,
          _ptr(out), _ptr(dmax), _stream())
    return out, dmax


# ----------------------------------------------------------------- convert --
def dense_to_band(A, kl, ku, AB=None, ldab=None):
    """Pack A into an (n, ldab) band tensor in xGBTRF layout."""
    _check(A, torch.float64, "A", 2)
    n = A.shape[0]
    if AB is None:
        ldab = ldab or 2 * kl + ku + 1
        AB = torch.empty((n, ldab), dtype=torch.float64, device=A.device)
    _check(AB, torch.float64, "AB", 2)
    _call("dense_to_band", _ptr(A), n, max(_ld(A), n, 1), kl, ku, _ptr(AB), max(_ld(AB), 1),
          _stream())
    return AB


def dense_to_band_batched(A, kl, ku, AB=None, ldab=None):
    _check(A, torch.float64, "A", 3)
    batch, n = A.shape[0], A.shape[1]
    if AB is None:
        ldab = ldab or 2 * kl + ku + 1
        AB = torch.empty((batch, n, ldab), dtype=torch.float64, device=A.device)
    _check(AB, torch.float64, "AB", 3)
    lda, ldab_ = max(_ld(A), n, 1), max(_ld(AB), 1)
    sA = A.stride(0) if batch > 1 else lda * n
    sAB = AB.stride(0) if batch > 1 else ldab_ * n
    _call("dense_to_band_batched", _ptr(A), n, lda, sA, kl, ku, _ptr(AB), ldab_, sAB, batch,
          _stream())
    return AB


# ------------------------------------------------------------------- getrf --
def _variant_code(variant):
    if variant is None:
        return 0
    if variant not in _VARIANT_CODES:
        raise ValueError(f"unknown variant {variant!r}; one of {sorted(_VARIANT_CODES)}")
    return _VARIANT_CODES[variant]


def band_getrf(AB, kl, ku, ipiv=None, info=None, variant=None):
    """In-place band LU; returns (ipiv int32 (n,), info int32 (1,)) on device.
    ``variant`` (a name from VARIANTS) forces a kernel through band_getrf_ex."""
    _check(AB, torch.float64, "AB", 2)
    n = AB.shape[0]
    if ipiv is None:
        ipiv = torch.empty(n, dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    ldab = max(_ld(AB), 1)
    if variant is None:
        _call("band_getrf", n, kl, ku, _ptr(AB), ldab, _ptr(ipiv), _ptr(info), _stream())
    else:
        _call("band_getrf_ex", n, kl, ku, _ptr(AB), ldab, ldab * n, _ptr(ipiv), n, _ptr(info), 1,
              _variant_code(variant), _stream())
    return ipiv, info


def band_getrf_batched(AB, kl, ku, ipiv=None, info=None, variant=None):
    """In-place batched band LU; returns (ipiv (batch, n), info (batch,))."""
    _check(AB, torch.float64, "AB", 3)
    batch, n = AB.shape[0], AB.shape[1]
    if ipiv is None:
        ipiv = torch.empty((batch, n), dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(batch, dtype=torch.int32, device=AB.device)
    ldab = max(_ld(AB), 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sP = ipiv.stride(0) if batch > 1 else n
    if variant is None:
        _call("band_getrf_batched", n, kl, ku, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(info),
              batch, _stream())
    else:
        _call("band_getrf_ex", n, kl, ku, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(info), batch,
              _variant_code(variant), _stream())
    return ipiv, info


def band_getrf_batched_noalloc(AB, kl, ku, ipiv, info):
    """band_getrf_batched without any device allocation, for callers that
    cannot allocate: the caller passes ipiv (batch, n) and info (batch,), and
    the wide-band kernel's scratch is the library's fixed per-device array."""
    _check(AB, torch.float64, "AB", 3)
    batch, n = AB.shape[0], AB.shape[1]
    ldab = max(_ld(AB), 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sP = ipiv.stride(0) if batch > 1 else n
    _call("band_getrf_batched_noalloc", n, kl, ku, _ptr(AB), ldab, sAB, _ptr(ipiv), sP,
          _ptr(info), batch, _stream())
    return ipiv, info


def band_getrf_variant(n, kl, ku, batch=1):
    v = _lib.band_getrf_variant(n, kl, ku, batch)
    if v < 0:
        raise BandLUError("band_getrf_variant", v)
    return VARIANTS[v]


# ------------------------------------------------------------------- getrs --
def _getrs_code(variant):
    if variant not in _GETRS_CODES:
        raise ValueError(f"unknown solve variant {variant!r}; one of {sorted(_GETRS_CODES)}")
    return _GETRS_CODES[variant]


def band_getrs(AB, kl, ku, ipiv, B, variant=None):
    """Solve in place; B has shape (nrhs, ldb) with B[k, i] = row i of rhs k.
    ``variant`` (a name from GETRS_VARIANTS) forces a kernel through band_getrs_ex."""
    _check(AB, torch.float64, "AB", 2)
    _check(ipiv, torch.int32, "ipiv", 1)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    nrhs = B.shape[0]
    ldb = max(_ld(B), n, 1)
    ldab = max(_ld(AB), 1)
    if variant is None:
        _call("band_getrs", n, kl, ku, nrhs, _ptr(AB), ldab, _ptr(ipiv), _ptr(B), ldb, _stream())
    else:
        _call("band_getrs_ex", n, kl, ku, nrhs, _ptr(AB), ldab, ldab * n, _ptr(ipiv), n, _ptr(B),
              ldb, ldb * nrhs, 1, _getrs_code(variant), _stream())
    return B


def band_getrs_variant(n, kl, ku, nrhs=1, batch=1):
    v = _lib.band_getrs_variant(n, kl, ku, nrhs, batch)
    if v < 0:
        raise BandLUError("band_getrs_variant", v)
    return GETRS_VARIANTS[v]


def band_getrs_batched(AB, kl, ku, ipiv, B, variant=None):
    """Batched solve in place; B has shape (batch, nrhs, ldb)."""
    _check(AB, torch.float64, "AB", 3)
    _check(ipiv, torch.int32, "ipiv", 2)
    _check(B, torch.float64, "B", 3)
    batch, n = AB.shape[0], AB.shape[1]
    nrhs = B.shape[1]
    ldab = max(_ld(AB), 1)
    ldb = max(_ld(B), n, 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sP = ipiv.stride(0) if batch > 1 else n
    sB = B.stride(0) if batch > 1 else ldb * nrhs
    if variant is None:
        _call("band_getrs_batched", n, kl, ku, nrhs, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(B),
              ldb, sB, batch, _stream())
    else:
        _call("band_getrs_ex", n, kl, ku, nrhs, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(B), ldb,
              sB, batch, _getrs_code(variant), _stream())
    return B


# ------------------------------------------------- fused detect + convert --
def band_detect_convert(A, kl_cap, ku_cap, AB=None, out=None):
    """Detection with caps and, in the same read, the band of the caps.

    Returns (out, AB): out = device int64 (kl, ku, exceeded); AB an (n, ldab)
    band array with ldab = 2*kl_cap + ku_cap + 1.  When exceeded is 0 the band
    of the detected (kl, ku) is ``band_view(AB, kl_cap, ku_cap, kl, ku)``."""
    _check(A, torch.float64, "A", 2)
    n = A.shape[0]
    if out is None:
        out = torch.empty(3, dtype=torch.int64, device=A.device)
    if AB is None:
        AB = torch.empty((n, 2 * kl_cap + ku_cap + 1), dtype=torch.float64, device=A.device)
    _check(AB, torch.float64, "AB", 2)
    _call("band_detect_convert", _ptr(A), n, max(_ld(A), n, 1), kl_cap, ku_cap, _ptr(out),
          _ptr(AB), max(_ld(AB), 1), _stream())
    return out, AB


def band_detect_convert_batched(A, kl_cap, ku_cap, AB=None, out=None, dmax=None):
    """Batched form; returns (out (batch, 3), dmax (3,), AB (batch, n, ldab))."""
    _check(A, torch.float64, "A", 3)
    batch, n = A.shape[0], A.shape[1]
    if out is None:
        out = torch.empty((batch, 3), dtype=torch.int64, device=A.device)
    if dmax is None:
        dmax = torch.empty(3, dtype=torch.int64, device=A.device)
    if AB is None:
        AB = torch.empty((batch, n, 2 * kl_cap + ku_cap + 1), dtype=torch.float64, device=A.device)
    _check(AB, torch.float64, "AB", 3)
    lda, ldab = max(_ld(A), n, 1), max(_ld(AB), 1)
    sA = A.stride(0) if batch > 1 else lda * n
    sAB = AB.stride(0) if batch > 1 else ldab * n
    _call("band_detect_convert_batched", _ptr(A), n, lda, sA, batch, kl_cap, ku_cap, _ptr(out),
          _ptr(dmax), _ptr(AB), ldab, sAB, _stream())
    return out, dmax, AB


def band_view(AB, kl_cap, ku_cap, kl, ku):
    """The xGBTRF band of (kl, ku) inside an array laid out for the caps: the
    same storage, starting kl_cap + ku_cap - kl - ku rows into each column
    (rows 0..2kl+ku of the view are the band; ldab stays that of AB)."""
    s = kl_cap + ku_cap - kl - ku
    return AB[..., s:s + 2 * kl + ku + 1]


# ------------------------------------------- triangular / diagonal solve --
def band_trsv(AB, kl, ku, B, info=None):
    """Listing 1's triangular / diagonal solve in place on B (nrhs, ldb) from
    the converted band (kl = 0 or ku = 0); returns info (device int32)."""
    _check(AB, torch.float64, "AB", 2)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    _call("band_trsv", n, kl, ku, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(B),
          max(_ld(B), n, 1), _ptr(info), _stream())
    return info


def band_trsv_batched(AB, kl, ku, B, info=None):
    _check(AB, torch.float64, "AB", 3)
    _check(B, torch.float64, "B", 3)
    batch, n = AB.shape[0], AB.shape[1]
    nrhs = B.shape[1]
    if info is None:
        info = torch.empty(batch, dtype=torch.int32, device=AB.device)
    ldab, ldb = max(_ld(AB), 1), max(_ld(B), n, 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sB = B.stride(0) if batch > 1 else ldb * nrhs
    _call("band_trsv_batched", n, kl, ku, nrhs, _ptr(AB), ldab, sAB, _ptr(B), ldb, sB, _ptr(info),
          batch, _stream())
    return info


# ---------------------------------------------------------- transposed solve --
def band_getrs_t(AB, kl, ku, ipiv, B):
    """Solve A^T X = B in place with band_getrf's factors; B is (nrhs, ldb)."""
    _check(AB, torch.float64, "AB", 2)
    _check(ipiv, torch.int32, "ipiv", 1)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    _call("band_getrs_t", n, kl, ku, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(ipiv), _ptr(B),
          max(_ld(B), n, 1), _stream())
    return B


def band_getrs_t_batched(AB, kl, ku, ipiv, B):
    _check(AB, torch.float64, "AB", 3)
    _check(ipiv, torch.int32, "ipiv", 2)
    _check(B, torch.float64, "B", 3)
    batch, n = AB.shape[0], AB.shape[1]
    nrhs = B.shape[1]
    ldab, ldb = max(_ld(AB), 1), max(_ld(B), n, 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sP = ipiv.stride(0) if batch > 1 else n
    sB = B.stride(0) if batch > 1 else ldb * nrhs
    _call("band_getrs_t_batched", n, kl, ku, nrhs, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(B),
          ldb, sB, batch, _stream())
    return B


# ----------------------------------------------------- rectangular band LU --
def band_getrf_mn(AB, m, kl, ku, ipiv=None, info=None):
    """LU of the m x n band matrix in AB (shape (n, ldab)); returns (ipiv, info)."""
    _check(AB, torch.float64, "AB", 2)
    n = AB.shape[0]
    if ipiv is None:
        ipiv = torch.empty(min(m, n), dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    _call("band_getrf_mn", m, n, kl, ku, _ptr(AB), max(_ld(AB), 1), _ptr(ipiv), _ptr(info),
          _stream())
    return ipiv, info


def band_getrf_mn_batched(AB, m, kl, ku, ipiv=None, info=None):
    _check(AB, torch.float64, "AB", 3)
    batch, n = AB.shape[0], AB.shape[1]
    if ipiv is None:
        ipiv = torch.empty((batch, min(m, n)), dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(batch, dtype=torch.int32, device=AB.device)
    ldab = max(_ld(AB), 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sP = ipiv.stride(0) if batch > 1 else min(m, n)
    _call("band_getrf_mn_batched", m, n, kl, ku, _ptr(AB), ldab, sAB, _ptr(ipiv), sP, _ptr(info),
          batch, _stream())
    return ipiv, info


# ---------------------------------------------------------- band Cholesky --
def band_is_symmetric(A, kd, flag=None):
    """Device int32: 1 if A(i, j) == A(j, i) for 0 < i - j <= kd."""
    _check(A, torch.float64, "A", 2)
    n = A.shape[0]
    if flag is None:
        flag = torch.empty(1, dtype=torch.int32, device=A.device)
    _call("band_is_symmetric", _ptr(A), n, max(_ld(A), n, 1), kd, _ptr(flag), _stream())
    return flag


def band_pbtrf(AB, kd, info=None):
    """Band Cholesky in place on the lower band AB (shape (n, ldab), element
    (i, j) at AB[j, i - j]); returns info (device int32)."""
    _check(AB, torch.float64, "AB", 2)
    n = AB.shape[0]
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    _call("band_pbtrf", n, kd, _ptr(AB), max(_ld(AB), 1), _ptr(info), _stream())
    return info


def band_pbtrf_batched(AB, kd, info=None):
    _check(AB, torch.float64, "AB", 3)
    batch, n = AB.shape[0], AB.shape[1]
    if info is None:
        info = torch.empty(batch, dtype=torch.int32, device=AB.device)
    ldab = max(_ld(AB), 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    _call("band_pbtrf_batched", n, kd, _ptr(AB), ldab, sAB, _ptr(info), batch, _stream())
    return info


def band_pbtrs(AB, kd, B):
    """Solve with band_pbtrf's factor in place on B (nrhs, ldb)."""
    _check(AB, torch.float64, "AB", 2)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    _call("band_pbtrs", n, kd, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(B), max(_ld(B), n, 1),
          _stream())
    return B


def band_pbtrs_batched(AB, kd, B):
    _check(AB, torch.float64, "AB", 3)
    _check(B, torch.float64, "B", 3)
    batch, n = AB.shape[0], AB.shape[1]
    nrhs = B.shape[1]
    ldab, ldb = max(_ld(AB), 1), max(_ld(B), n, 1)
    sAB = AB.stride(0) if batch > 1 else ldab * n
    sB = B.stride(0) if batch > 1 else ldb * nrhs
    _call("band_pbtrs_batched", n, kd, nrhs, _ptr(AB), ldab, sAB, _ptr(B), ldb, sB, batch,
          _stream())
    return B


# --------------------------------------------------- factor + solve (xGBSV) --
def band_gbsv(AB, kl, ku, B, ipiv=None, info=None):
    """band_getrf then band_getrs in one call (the forward substitution fused
    into the persistent wide-band LU where that kernel runs); B (nrhs, ldb) is
    overwritten with X.  Returns (ipiv, info)."""
    _check(AB, torch.float64, "AB", 2)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    if ipiv is None:
        ipiv = torch.empty(n, dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    _call("band_gbsv", n, kl, ku, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(ipiv), _ptr(B),
          max(_ld(B), n, 1), _ptr(info), _stream())
    return ipiv, info


def band_gbsv_lu(AB, kl, ku, B, ipiv=None, info=None):
    """The first half of band_gbsv: band_getrf, and B <- L^-1 P B (inside the
    persistent wide-band launch where it runs, and inside the 64-lane window
    kernel's steps for one right-hand side with 1 <= kl <= 6).  Returns
    (ipiv, info)."""
    _check(AB, torch.float64, "AB", 2)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    if ipiv is None:
        ipiv = torch.empty(n, dtype=torch.int32, device=AB.device)
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=AB.device)
    _call("band_gbsv_lu", n, kl, ku, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(ipiv), _ptr(B),
          max(_ld(B), n, 1), _ptr(info), _stream())
    return ipiv, info


def band_gbsv_back(AB, kl, ku, B):
    """The second half of band_gbsv: B <- U^-1 B from the factors."""
    _check(AB, torch.float64, "AB", 2)
    _check(B, torch.float64, "B", 2)
    n = AB.shape[0]
    _call("band_gbsv_back", n, kl, ku, B.shape[0], _ptr(AB), max(_ld(AB), 1), _ptr(B),
          max(_ld(B), n, 1), _stream())
    return B
