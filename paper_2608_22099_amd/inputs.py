"""Seeded synthetic inputs: banded matrices stored densely, and right-hand sides.

This module holds no arithmetic of the method.  It only draws random numbers
and places them, so both the HIP path and the CPU oracle can be fed the same
bytes.  It imports nothing but numpy.

Storage convention: a numpy array ``T`` of shape (n, n) in C order holds the
column-major matrix A as ``T[j, i] = A[i, j]`` (row j of T is column j of A).

Recipe (one per named workload):
  * RNG = numpy.random.Generator(PCG64(seed));
  * in-band values are drawn in column-major in-band order: column j ascending,
    then row i ascending from max(0, j-ku) to min(n-1, j+kl);
  * a diagonal shift, where the workload has one, is added after drawing;
  * every out-of-band entry is exactly +0.0;
  * right-hand sides are iid N(0,1) with seed = base seed + 500000 (+ batch
    index for batched workloads).
The paper benchmarks randomly generated banded matrices converted to dense
storage (Sec. IV); these generators stand in for them.
"""
from __future__ import annotations

import numpy as np

RHS_SEED_OFFSET = 500_000

# Named workloads: dense-stored banded fp64 matrices.
WORKLOADS = {
    "n1000_kl3_ku3": dict(n=1000, kl=3, ku=3, dist="normal", shift=0.0, seed=1_000_000,
                          batch=1, nrhs=1),
    "n8192_kl16_ku16": dict(n=8192, kl=16, ku=16, dist="normal", shift=64.0, seed=2_000_000,
                            batch=1, nrhs=1),
    "n16384_kl2_ku64": dict(n=16384, kl=2, ku=64, dist="uniform", shift=0.0, seed=3_000_000,
                            batch=1, nrhs=1),
    "batch4096_n256_kl4_ku4": dict(n=256, kl=4, ku=4, dist="normal", shift=0.0, seed=4_000_000,
                                   batch=4096, nrhs=1),
    "n32768_kl256_ku256": dict(n=32768, kl=256, ku=256, dist="normal", shift=1024.0,
                               seed=5_000_000, batch=1, nrhs=1),
}


def _draw(rng, dist, count):
    if dist == "normal":
        return rng.standard_normal(count)
    if dist == "uniform":
        return rng.uniform(-1.0, 1.0, count)
    raise ValueError(f"unknown distribution {dist!r}")


def band_index(n, kl, ku):
    """(j, i) index arrays of the in-band entries in column-major in-band order."""
    offs = np.arange(-ku, kl + 1, dtype=np.int64)
    j = np.repeat(np.arange(n, dtype=np.int64), offs.size)
    i = j + np.tile(offs, n)
    keep = (i >= 0) & (i < n)
    return j[keep], i[keep]


def banded_dense(n, kl, ku, seed, dist="normal", shift=0.0, out=None, check=True):
    """Dense-stored banded matrix with exact bandwidths (kl, ku).

    ``out`` may be a preallocated float64 array of shape (n, lda), lda >= n;
    it is zeroed first.  Returns the (n, lda) array.
    """
    if out is None:
        # zeroed by one sequential pass: pages touched first by the scattered
        # band writes below are far slower to map than pages touched in order
        out = np.empty((n, n), dtype=np.float64)
        out.fill(0.0)
    else:
        if out.shape[0] != n or out.shape[1] < n or out.dtype != np.float64:
            raise ValueError("out must be float64 of shape (n, lda >= n)")
        out[...] = 0.0
    if n == 0:
        return out
    rng = np.random.Generator(np.random.PCG64(seed))
    j, i = band_index(n, kl, ku)
    out[j, i] = _draw(rng, dist, j.size)
    if shift:
        d = np.arange(n)
        out[d, d] += shift
    if check:
        if kl > 0:
            d = np.arange(n - kl)
            assert np.any(out[d, d + kl] != 0.0), "lowest diagonal is empty"
        if ku > 0:
            d = np.arange(ku, n)
            assert np.any(out[d, d - ku] != 0.0), "highest diagonal is empty"
    return out


def column_dominant(T):
    """True if every column of A (rows of T) is strictly diagonally dominant."""
    n = T.shape[0]
    a = np.abs(T[:, :n])
    diag = np.diagonal(a).copy()
    return bool(np.all(a.sum(axis=1) - diag < diag))


def workload_matrix(name, index=0, out=None):
    """Matrix ``index`` of a named workload (index is the batch position)."""
    w = WORKLOADS[name]
    return banded_dense(w["n"], w["kl"], w["ku"], w["seed"] + index, w["dist"], w["shift"],
                        out=out)


def workload_rhs(name, index=0, nrhs=None):
    """Right-hand sides (nrhs, n) for matrix ``index`` of a named workload."""
    w = WORKLOADS[name]
    k = w["nrhs"] if nrhs is None else nrhs
    rng = np.random.Generator(np.random.PCG64(w["seed"] + RHS_SEED_OFFSET + index))
    return rng.standard_normal((k, w["n"]))


def workload_batch(name, count=None, out=None):
    """Stack of ``count`` matrices of a batched workload, shape (count, n, n)."""
    w = WORKLOADS[name]
    count = w["batch"] if count is None else count
    n = w["n"]
    if out is None:
        out = np.zeros((count, n, n), dtype=np.float64)
    for b in range(count):
        banded_dense(n, w["kl"], w["ku"], w["seed"] + b, w["dist"], w["shift"], out=out[b])
    return out


def random_case(seed, n_max=40, special=False, lda_pad=0):
    """A random small test case: random n, kl, ku, optional padding and specials.

    Returns (T, kl, ku) with T of shape (n, n + lda_pad).  With ``special``,
    some in-band entries are replaced by -0.0, +0.0 and whole columns may be
    zeroed, so the detected bandwidths can be smaller than (kl, ku).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    n = int(rng.integers(1, n_max + 1))
    kl = int(rng.integers(0, n))
    ku = int(rng.integers(0, n))
    T = np.zeros((n, n + lda_pad), dtype=np.float64)
    if lda_pad:
        T[:, n:] = rng.standard_normal((n, lda_pad))  # padding rows must be ignored
    j, i = band_index(n, kl, ku)
    T[j, i] = rng.standard_normal(j.size)
    if special and j.size:
        pick = rng.random(j.size)
        T[j[pick < 0.1], i[pick < 0.1]] = -0.0
        T[j[(pick >= 0.1) & (pick < 0.2)], i[(pick >= 0.1) & (pick < 0.2)]] = 0.0
        if n > 2 and rng.random() < 0.5:
            T[int(rng.integers(0, n)), :n] = 0.0
    return T, kl, ku
