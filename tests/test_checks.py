"""The tolerance rules the GPU parity tests use, pinned on the CPU against the
oracle itself: a perturbation within the tolerance passes, one beyond it (or a
zero that is not zero) fails, and the band mat-vec equals the dense product."""
import numpy as np
import pytest

import oracle
from checks import assert_factors_close, assert_solve_residual, band_matvec
from paper_2608_22099_amd import inputs


def factored(n, kl, ku, seed):
    T = inputs.banded_dense(n, kl, ku, seed, check=False)
    AB, _ = oracle.dense_to_band(T, kl, ku)
    AB0 = AB.copy()
    ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
    return T, AB0, AB, ipiv


def test_tolerance_rule_accepts_rounding_and_rejects_errors():
    n, kl, ku = 120, 7, 5
    _, _, AB, _ = factored(n, kl, ku, 3)
    assert assert_factors_close(AB, AB.copy(), kl, ku, "self") == 0
    kv = kl + ku
    g = AB.copy()
    g[50, kv] *= 1 + 1e-13          # a diagonal entry of U, within 1e-10
    g[60, kv + 2] *= 1 + 1e-12      # a multiplier, within 1e-10
    assert_factors_close(g, AB, kl, ku, "rounding")
    for j, r, f in [(50, kv, 1 + 1e-8), (60, kv + 2, -1.0)]:
        bad = AB.copy()
        bad[j, r] *= f
        with pytest.raises(AssertionError):
            assert_factors_close(bad, AB, kl, ku, "planted")
    bad = AB.copy()
    zero = np.argwhere((AB == 0.0) & (np.arange(AB.shape[1])[None, :] < kv))
    j, r = zero[len(zero) // 2]
    if r - kv + j >= 0:
        bad[j, r] = 1e-300              # an exact zero of U that is not zero
        with pytest.raises(AssertionError):
            assert_factors_close(bad, AB, kl, ku, "zero")


def test_band_matvec_and_residual():
    n, kl, ku = 90, 4, 9
    T, AB0, AB, ipiv = factored(n, kl, ku, 5)
    x = np.random.default_rng(0).standard_normal(n)
    A = T.T  # T[j, i] = A[i, j]
    assert np.allclose(band_matvec(AB0, kl, ku, x), A @ x, rtol=1e-13, atol=1e-12)
    b = np.random.default_rng(1).standard_normal((1, n))
    xs = oracle.gbtrs(AB, kl, ku, ipiv, b.copy())[0]
    assert_solve_residual(AB0, kl, ku, xs, b[0], "oracle solve")
    with pytest.raises(AssertionError):
        assert_solve_residual(AB0, kl, ku, xs * (1 + 1e-6), b[0], "perturbed solve")
