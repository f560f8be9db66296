"""Host policy of Listing 2 on the CPU: the Sec. II-B constraints as
operation counts and from a cost model, and the early-exit caps they give
(no GPU: the model here is written by hand)."""
import numpy as np

from paper_2608_22099_amd import inputs, policy


def test_op_count_constraints_on_workloads():
    for w in inputs.WORKLOADS.values():
        assert policy.speedup_predicate(w["n"], w["kl"], w["ku"])
        assert policy.slowdown_constraint(w["n"])
    assert not policy.speedup_predicate(1000, 999, 999)  # dense: f > F


def test_caps_bound_the_banded_branch():
    """Every (kl, ku) that satisfies the constraint lies within the caps, and
    the caps themselves (with the other bandwidth zero) satisfy it."""
    rng = np.random.default_rng(0)
    for n in (10, 300, 4096, 32768):
        kl_cap, ku_cap = policy.band_caps(n)
        if kl_cap >= 0:
            assert policy.speedup_predicate(n, kl_cap, 0)
            assert not policy.speedup_predicate(n, kl_cap + 1, 0)
        if ku_cap >= 0:
            assert policy.speedup_predicate(n, 0, ku_cap)
        for _ in range(200):
            kl, ku = (int(v) for v in rng.integers(0, n, 2))
            if policy.speedup_predicate(n, kl, ku):
                assert kl_cap < 0 or kl <= kl_cap
                assert ku_cap < 0 or ku <= ku_cap


def test_model_predicate():
    m = policy.CostModel(detect_bps=5e12, convert_bps=4e12, call_s=5e-6,
                         lu_probe={(4, 4): 300e-9, (64, 64): 2e-6, (256, 256): 40e-6},
                         lu_probe_n=2048, dense_a=1e-3, dense_b=1e-12)
    I, C, f, F = m.times(8192, 3, 3)
    assert f == m.call_s + 300e-9 * 8192 and abs(F - (1e-3 + 8192.0 ** 3 * 1e-12)) < 1e-12
    assert policy.speedup_predicate(8192, 16, 16, m)
    assert not policy.speedup_predicate(2048, 1000, 1000, m)
    kl_cap, _ = policy.band_caps(8192, m)
    assert 0 < kl_cap < 8191 and not policy.speedup_predicate(8192, kl_cap + 1, 0, m)
