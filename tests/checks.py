"""Comparison rules shared by the GPU parity tests (no tests here).

Factors that are not bitwise those of the unblocked algorithm (the matrix-core
variant sums its updates in another order) are held to the method's tolerance:
every factor entry within relative error 1e-10 of the oracle's, where an
entry that fails only because the oracle value is small against its column
(cancellation) passes against 1e-10 times the largest magnitude of that part
(U or L) of the column and is counted; oracle zeros must be exact zeros; and
the backward error ||PA - LU||_F / (||A||_F n eps) is at most 10.
"""
import numpy as np

import oracle

RTOL = 1e-10
BACKWARD_BOUND = 10.0


def bits(x):
    return np.ascontiguousarray(x).view(np.uint64)


def factor_slots(n, kl, ku, ldab):
    """Masks (n, ldab) of the band slots inside the matrix that hold U (rows
    0..kl+ku of column j) and the multipliers of L (rows kl+ku+1..2kl+ku)."""
    kv = kl + ku
    j = np.arange(n)[:, None]
    r = np.arange(ldab)[None, :]
    i = r - kv + j
    inside = (i >= 0) & (i < n)
    return inside & (r <= kv), inside & (r > kv) & (r <= kv + kl)


def assert_factors_close(g, o, kl, ku, what, rtol=RTOL):
    """Tolerance parity of band factors g (GPU) and o (oracle), both (n, ldab).
    Returns the number of entries that passed only on the column scale."""
    g = np.ascontiguousarray(g)
    o = np.ascontiguousarray(o)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    n, ldab = o.shape
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(g)), f"{what}: non-finite factors"
    U, L = factor_slots(n, kl, ku, ldab)
    outside = ~(U | L)
    assert np.array_equal(bits(g)[outside], bits(o)[outside]), f"{what}: slots outside the factors"
    diff = np.abs(g - o)
    fallback = 0
    for part, name in ((U, "U"), (L, "L")):
        zero = part & (o == 0.0)
        nz = np.count_nonzero(g[zero])
        assert nz == 0, f"{what}: {nz} exact zeros of {name} are not zero on the GPU"
        scale = np.where(part, np.abs(o), 0.0).max(axis=1, keepdims=True)
        rel_ok = diff <= rtol * np.abs(o)
        col_ok = diff <= rtol * scale
        bad = part & ~rel_ok & ~col_ok
        if bad.any():
            j, r = (int(v[0]) for v in np.nonzero(bad))
            raise AssertionError(f"{what}: {np.count_nonzero(bad)} {name} entries beyond tolerance, "
                                 f"first column {j} slot {r}: gpu={g[j, r]!r} oracle={o[j, r]!r}")
        fallback += int(np.count_nonzero(part & ~rel_ok & col_ok))
    return fallback


def assert_backward_error(AB0, ABf, kl, ku, ipiv, what):
    e = oracle.band_backward_error(AB0, ABf, kl, ku, ipiv)
    assert e <= BACKWARD_BOUND, f"{what}: backward error {e}"
    return e


def band_matvec(AB0, kl, ku, x):
    """y = A x for the band in AB0 (n, ldab), xGBTRF layout at rows kl.. ."""
    n = AB0.shape[0]
    kv = kl + ku
    y = np.zeros(n)
    for d in range(-ku, kl + 1):  # d = i - j
        j = np.arange(max(0, -d), min(n, n - d))
        y[j + d] += AB0[j, kv + d] * x[j]
    return y


def assert_solve_residual(AB0, kl, ku, x, b, what):
    """||A x - b||_inf / (||A||_inf ||x||_inf n eps) <= 10."""
    n = AB0.shape[0]
    r = band_matvec(AB0, kl, ku, x) - b
    anorm = band_matvec(np.abs(AB0), kl, ku, np.ones(n)).max()
    e = np.abs(r).max() / (anorm * np.abs(x).max() * n * np.finfo(float).eps)
    assert e <= BACKWARD_BOUND, f"{what}: solve residual {e}"
    return e
