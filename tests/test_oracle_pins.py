"""Pins for the CPU oracle: checks against facts that do not come from the
oracle itself (brute force, closed forms, special cases, a library routine,
invariants of the method, numbers printed in the paper).  CPU only.
"""
import math
import os

import numpy as np
import pytest
import scipy.linalg.lapack as lapack

import oracle
from paper_2608_22099_amd import inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# --------------------------------------------------------------------------
# helpers written independently of the oracle (plain numpy)
# --------------------------------------------------------------------------
def np_bandwidths(T):
    """Brute force with numpy: max(i-j), max(j-i) over entries != 0."""
    n = T.shape[0]
    jj, ii = np.nonzero(T[:, :n] != 0.0)  # T[j, i] = A[i, j]
    if jj.size == 0:
        return 0, 0
    return int(max(0, (ii - jj).max())), int(max(0, (jj - ii).max()))


def np_band_to_dense(AB, kl, ku, n):
    """Unpack the xGBTRF-layout band (AB[j, r]) of the ORIGINAL matrix into T[j, i]."""
    T = np.zeros((n, n))
    kv = kl + ku
    for j in range(n):
        for i in range(max(0, j - ku), min(n - 1, j + kl) + 1):
            T[j, i] = AB[j, kv + i - j]
    return T


def random_band(n, kl, ku, seed, lda_pad=0):
    T = np.zeros((n, n + lda_pad))
    rng = np.random.default_rng(seed)
    j, i = inputs.band_index(n, kl, ku)
    T[j, i] = rng.standard_normal(j.size)
    if lda_pad:
        T[:, n:] = 7.0
    return T


def bits(x):
    return np.ascontiguousarray(x).view(np.uint64)


# --------------------------------------------------------------------------
# detection (Sec. II-A step 1; Listing 1 element inspection; Listing 2)
# --------------------------------------------------------------------------
class TestDetect:
    def test_special_cases(self):
        n = 9
        Z = np.zeros((n, n))
        assert oracle.detect(Z)[:3] == (0, 0, 0)
        D = np.diag(np.arange(1.0, n + 1))
        assert oracle.detect(D)[:2] == (0, 0)
        full = np.ones((n, n))
        assert oracle.detect(full)[:2] == (n - 1, n - 1)
        A = np.tril(np.ones((n, n)))      # as a matrix A (row-major view of A)
        T = np.ascontiguousarray(A.T)     # column-major storage of A
        assert oracle.detect(T)[:2] == (n - 1, 0)  # full lower triangle
        T = np.ascontiguousarray(np.triu(np.ones((n, n))).T)
        assert oracle.detect(T)[:2] == (0, n - 1)  # full upper triangle
        for (i, j) in [(0, 0), (5, 1), (1, 7), (8, 0), (0, 8)]:
            S = np.zeros((n, n))
            S[j, i] = 3.0
            assert oracle.detect(S)[:2] == (max(0, i - j), max(0, j - i))

    def test_zero_signs_nan_inf_subnormal(self):
        n = 6
        S = np.zeros((n, n))
        S[0, 4] = -0.0           # A[4, 0] = -0.0 counts as zero
        assert oracle.detect(S)[:2] == (0, 0)
        S[0, 3] = np.nan         # A[3, 0] = NaN counts as nonzero
        assert oracle.detect(S)[:2] == (3, 0)
        S[5, 1] = np.inf         # A[1, 5]
        assert oracle.detect(S)[:2] == (3, 4)
        S2 = np.zeros((n, n))
        S2[2, 0] = 5e-324        # subnormal is nonzero
        assert oracle.detect(S2)[:2] == (0, 2)

    @pytest.mark.parametrize("seed", range(40))
    def test_random_vs_numpy_bruteforce(self, seed):
        T, kl, ku = inputs.random_case(seed, n_max=30, special=True, lda_pad=seed % 3)
        n = T.shape[0]
        kl_o, ku_o, ex, cnt = oracle.detect(T)
        assert (kl_o, ku_o) == np_bandwidths(T[:, :n])
        assert kl_o <= kl and ku_o <= ku
        assert cnt == n * n
        assert ex == 0

    def test_listing1_triangular_equivalences(self):
        # istril(A) <=> ku == 0 and istriu(A) <=> kl == 0 (Listing 1 branches)
        for seed in range(20):
            T, _, _ = inputs.random_case(100 + seed, n_max=12, special=True)
            n = T.shape[0]
            A = T[:, :n].T
            kl, ku, _, _ = oracle.detect(T)
            assert (ku == 0) == bool(np.all(np.triu(A, 1) == 0))
            assert (kl == 0) == bool(np.all(np.tril(A, -1) == 0))

    @pytest.mark.parametrize("name", list(inputs.WORKLOADS))
    def test_generator_known_bandwidths(self, name):
        w = inputs.WORKLOADS[name]
        n = min(w["n"], 1000)  # same recipe, CPU-sized
        kl, ku = min(w["kl"], n - 1), min(w["ku"], n - 1)
        T = inputs.banded_dense(n, kl, ku, w["seed"], w["dist"], w["shift"])
        assert oracle.detect(T)[:2] == (kl, ku)

    def test_caps(self):
        T = random_band(20, 3, 5, 1)
        assert oracle.detect(T, 3, 5)[2] == 0
        assert oracle.detect(T, 2, -1)[2] == 1
        assert oracle.detect(T, -1, 4)[2] == 1
        assert oracle.detect(T, -1, -1)[2] == 0
        assert oracle.detect(T, 100, 100)[:3] == (3, 5, 0)

    def test_empty(self):
        T = np.zeros((0, 1))
        assert oracle.detect(T) == (0, 0, 0, 0)


# --------------------------------------------------------------------------
# conversion (Sec. II-A step 2; Listing 2 dense -> band)
# --------------------------------------------------------------------------
class TestConvert:
    @pytest.mark.parametrize("seed", range(30))
    def test_round_trip_and_layout(self, seed):
        T, kl, ku = inputs.random_case(200 + seed, n_max=25, special=True, lda_pad=seed % 2)
        n = T.shape[0]
        ldab = 2 * kl + ku + 1 + (seed % 3)
        AB, written = oracle.dense_to_band(T, kl, ku, ldab=ldab)
        assert written == (2 * kl + ku + 1) * n
        # bitwise round trip (keeps -0.0)
        back = np_band_to_dense(AB, kl, ku, n)
        assert np.array_equal(bits(back), bits(T[:, :n]))
        # fill rows and out-of-matrix slots are +0.0 bit patterns
        kv = kl + ku
        for j in range(n):
            for r in range(2 * kl + ku + 1):
                i = r - kv + j
                if r < kl or i < 0 or i >= n:
                    assert bits(AB[j, r:r + 1])[0] == 0
            # rows beyond 2kl+ku are untouched (sentinel NaN from the wrapper)
            assert np.all(np.isnan(AB[j, 2 * kl + ku + 1:]))

    def test_nan_payload_kept(self):
        T = np.zeros((3, 3))
        payload = np.array([0x7FF8_0000_0000_1234], dtype=np.uint64).view(np.float64)[0]
        T[1, 1] = payload
        AB, _ = oracle.dense_to_band(T, 1, 1)
        assert bits(AB[1, 2:3])[0] == 0x7FF8_0000_0000_1234

    def test_paper_memory_figures_fix_ldab(self):
        """Sec. IV-B prints 763.02 MiB (dense) and 68.97 MiB (structure-aware)
        for n = 1e4 with 100 sub- and 100 super-diagonals.  Three band arrays
        of the xGBTRF leading dimension 2kl+ku+1 plus an int64 pivot vector
        reproduce the second figure; one dense copy plus the pivots the first."""
        g = {}
        with open(os.path.join(GOLDEN, "paper_sec4b_memory.txt")) as f:
            for line in f:
                if line.strip() and not line.startswith("#"):
                    k, v = line.split("=")
                    g[k.strip()] = float(v)
        n, kl, ku = int(g["n"]), int(g["kl"]), int(g["ku"])
        T = np.zeros((4, 4))
        AB, _ = oracle.dense_to_band(T, 2, 1)
        assert AB.shape[1] == 2 * 2 + 1 + 1
        ldab = 2 * kl + ku + 1
        mib = 1024.0 ** 2
        assert round((3 * ldab * n * 8 + n * 8) / mib, 2) == g["structured_mib"]
        assert round((n * n * 8 + n * 8) / mib, 2) == g["dense_mib"]


# --------------------------------------------------------------------------
# banded LU (Sec. III-A, xGBTRF)
# --------------------------------------------------------------------------
def band_lu(T, kl, ku):
    AB, _ = oracle.dense_to_band(T, kl, ku)
    AB0 = AB.copy()
    ipiv, info, flops = oracle.gbtrf(AB, kl, ku)
    return AB0, AB, ipiv, info, flops


class TestBandLU:
    @pytest.mark.parametrize("seed", range(60))
    def test_bruteforce_dense_gepp(self, seed):
        """Dense GEPP on the same banded matrix gives identical pivots and U,
        and its L equals the band multipliers after the later interchanges."""
        rng = np.random.default_rng(seed)
        n = int(rng.integers(1, 13))
        kl, ku = int(rng.integers(0, n)), int(rng.integers(0, n))
        T = random_band(n, kl, ku, 1000 + seed, lda_pad=int(rng.integers(0, 3)))
        AB0, AB, ipiv, info, _ = band_lu(T, kl, ku)
        D = T.copy()
        dpiv, dinfo = oracle.dense_gepp(D)
        assert info == dinfo == 0
        assert np.array_equal(ipiv, dpiv)
        kv = kl + ku
        A_lu = D[:, :n].T  # dense factors, A_lu[i, c]
        for c in range(n):
            for i in range(c + 1):
                u_band = AB[c, kv + i - c] if c - i <= kv else 0.0
                assert A_lu[i, c] == u_band, (i, c)
        for j in range(n):
            v = np.zeros(n)
            km = min(kl, n - 1 - j)
            v[j + 1:j + 1 + km] = AB[j, kv + 1:kv + 1 + km]
            for k in range(j + 1, n):
                q = ipiv[k] - 1
                v[k], v[q] = v[q], v[k]
            assert np.array_equal(v[j + 1:], A_lu[j + 1:, j]), j

    def test_hand_example(self):
        """3x3, kl = ku = 1, worked by hand (tests/golden/hand_3x3.txt)."""
        A = np.array([[1.0, 2.0, 0.0], [5.0, 1.0, 3.0], [0.0, 4.0, 1.0]])
        T = np.ascontiguousarray(A.T)
        _, AB, ipiv, info, _ = band_lu(T, 1, 1)
        assert info == 0
        assert list(ipiv) == [2, 3, 3]
        kv = 2
        U = [[AB[c, kv + i - c] if i <= c else 0.0 for c in range(3)] for i in range(3)]
        np.testing.assert_allclose(U, [[5, 1, 3], [0, 4, 1], [0, 0, -1.05]], rtol=1e-15, atol=1e-15)
        assert AB[2, 0] == 3.0          # fill U(0, 2) lands in AB row 0
        np.testing.assert_allclose([AB[0, kv + 1], AB[1, kv + 1]], [0.2, 0.45], rtol=1e-15)

    def test_tridiagonal_toeplitz_closed_form(self):
        """[-1, 4, -1]: no pivoting, u_k = 4 - 1/u_{k-1} has the closed form
        u_k = (a^(k+2) - b^(k+2)) / (a^(k+1) - b^(k+1)), a, b = 2 +- sqrt(3)."""
        n = 60
        A = 4 * np.eye(n) - np.eye(n, k=1) - np.eye(n, k=-1)
        _, AB, ipiv, info, _ = band_lu(np.ascontiguousarray(A.T), 1, 1)
        assert info == 0 and np.array_equal(ipiv, np.arange(1, n + 1))
        a, b = 2 + math.sqrt(3), 2 - math.sqrt(3)
        for k in range(n):
            u = (a ** (k + 2) - b ** (k + 2)) / (a ** (k + 1) - b ** (k + 1))
            assert abs(AB[k, 2] - u) <= 4e-15 * u
            if k > 0:
                assert abs(AB[k - 1, 3] - (-1.0 / u_prev)) <= 4e-15
            u_prev = u
        assert np.all(AB[:, 0] == 0.0)  # no fill without pivoting

    @pytest.mark.parametrize("name", list(inputs.WORKLOADS))
    def test_dominant_means_identity_pivots(self, name):
        """Strict column diagonal dominance keeps GEPP on the diagonal (and
        survives in the Schur complement): ipiv = identity and no fill."""
        w = inputs.WORKLOADS[name]
        if w["shift"] == 0.0:
            pytest.skip("workload is not diagonally dominant by construction")
        n = 700
        T = inputs.banded_dense(n, w["kl"], w["ku"], w["seed"], w["dist"], w["shift"])
        assert inputs.column_dominant(T)
        _, AB, ipiv, info, _ = band_lu(T, w["kl"], w["ku"])
        assert info == 0 and np.array_equal(ipiv, np.arange(1, n + 1))
        assert np.all(AB[:, :w["kl"]] == 0.0)

    def test_fill_rows_not_read(self):
        """Band rows 0..kl-1 are workspace for fill: their entry contents must
        not matter (xGBTRF zeroes them before use)."""
        for seed in range(10):
            T = random_band(40, 3, 4, 70 + seed)
            AB, _ = oracle.dense_to_band(T, 3, 4)
            AB2 = AB.copy()
            AB2[:, :3] = np.nan
            p1, i1, _ = oracle.gbtrf(AB, 3, 4)
            p2, i2, _ = oracle.gbtrf(AB2, 3, 4)
            kv = 7
            for j in range(40):  # out-of-matrix corner slots keep what was there
                for r in range(3):
                    if r - kv + j < 0:
                        AB2[j, r] = AB[j, r]
            assert np.array_equal(p1, p2) and i1 == i2
            assert np.array_equal(bits(AB), bits(AB2))

    def test_singular_info(self):
        n = 10
        for k in [0, 3, 9]:
            T = random_band(n, 2, 2, 50 + k)
            T[k, :] = 0.0  # zero column k of A
            _, _, ipiv, info, _ = band_lu(T, 2, 2)
            assert info == k + 1
            assert ipiv[k] == k + 1
        _, AB, ipiv, info, _ = band_lu(np.zeros((5, 5)), 1, 2)
        assert info == 1 and np.array_equal(ipiv, np.arange(1, 6))
        assert np.all(AB == 0.0)

    def test_subnormal_pivot_divides(self):
        """A pivot below DBL_MIN is divided into the column instead of being
        inverted (1/p would overflow to Inf).  The multipliers and the Schur
        complement are exact by hand: 2t/4t = 0.5, 3 - 0.5*2 = 2, and t/3t is
        the correctly rounded 1/3 (t = 2^-1074, the smallest subnormal).
        Checked on the band routine and on the dense brute force."""
        t = math.ldexp(1.0, -1074)
        third = np.array([0x3FD5555555555555], dtype=np.uint64).view(np.float64)[0]
        for p, a, l_want, u22_want in [(4 * t, 2 * t, 0.5, 2.0), (3 * t, t, third, 3.0 - third * 2.0)]:
            assert 0.0 < p < np.finfo(float).tiny
            A = np.array([[p, 2.0], [a, 3.0]])
            T = np.ascontiguousarray(A.T)
            _, AB, ipiv, info, _ = band_lu(T, 1, 1)
            assert info == 0 and list(ipiv) == [1, 2]
            assert AB[0, 3] == l_want and bits(AB[0, 3:4])[0] == bits(np.array([l_want]))[0]
            assert AB[1, 2] == u22_want
            assert AB[0, 2] == p and AB[1, 1] == 2.0
            D = T.copy()
            dpiv, dinfo = oracle.dense_gepp(D)
            assert dinfo == 0 and list(dpiv) == [1, 2]
            assert D[0, 1] == l_want and D[1, 1] == u22_want
        # a pivot exactly at DBL_MIN is inverted (2^1022 is finite): 1/DBL_MIN
        # times DBL_MIN/2 is exactly 0.5 either way, and the branch boundary
        # must not send it to Inf
        m = np.finfo(float).tiny
        T = np.ascontiguousarray(np.array([[m, 1.0], [m / 2, 1.0]]).T)
        _, AB, ipiv, info, _ = band_lu(T, 1, 1)
        assert AB[0, 3] == 0.5 and AB[1, 2] == 0.5

    def test_nan_pivot_convention(self):
        """i_amax: a NaN in first position is taken, later NaNs are never taken."""
        A = np.array([[np.nan, 1.0], [3.0, 1.0]])
        _, AB, ipiv, info, _ = band_lu(np.ascontiguousarray(A.T), 1, 1)
        assert ipiv[0] == 1
        A = np.array([[1.0, 1.0, 0.0], [np.nan, 1.0, 1.0], [2.0, 1.0, 1.0]])
        _, AB, ipiv, info, _ = band_lu(np.ascontiguousarray(A.T), 2, 1)
        assert ipiv[0] == 3
        A = np.array([[2.0, 1.0], [-2.0, 1.0]])  # tie: first index wins
        _, AB, ipiv, info, _ = band_lu(np.ascontiguousarray(A.T), 1, 1)
        assert ipiv[0] == 1

    @pytest.mark.parametrize("seed", range(25))
    def test_scipy_dgbtrf(self, seed):
        """LAPACK dgbtrf (a library pin): same pivots, factors to rounding."""
        rng = np.random.default_rng(seed)
        n = int(rng.integers(2, 120))
        kl, ku = int(rng.integers(0, min(n, 12))), int(rng.integers(0, min(n, 12)))
        T = random_band(n, kl, ku, 3000 + seed)
        AB0, AB, ipiv, info, _ = band_lu(T, kl, ku)
        lu, piv, linfo = lapack.dgbtrf(np.asfortranarray(AB0.T), kl, ku)
        assert linfo == info == 0
        assert np.array_equal(piv + 1, ipiv)
        ref = lu.T
        assert np.allclose(AB[:, :2 * kl + ku + 1], ref[:, :2 * kl + ku + 1], rtol=1e-12, atol=1e-12)

    def test_fill_bound_and_flop_bound(self):
        for seed in range(20):
            rng = np.random.default_rng(seed)
            n = int(rng.integers(5, 200))
            kl, ku = int(rng.integers(0, 8)), int(rng.integers(0, 8))
            kl, ku = min(kl, n - 1), min(ku, n - 1)
            T = random_band(n, kl, ku, 4000 + seed)
            AB0, AB, ipiv, info, flops = band_lu(T, kl, ku)
            assert flops <= 2 * n * kl * (kl + ku + 1)
            assert 0.0 <= oracle.band_backward_error(AB0, AB, kl, ku, ipiv) <= 10.0
            # multipliers bounded by 1 in magnitude (partial pivoting)
            kv = kl + ku
            assert np.all(np.abs(AB[:, kv + 1:2 * kl + ku + 1]) <= 1.0)

    def test_flops_linear_in_n(self):
        """f(N) = O(N * P * Q) at fixed bandwidths (Sec. III-A)."""
        counts = []
        for n in [1024, 2048, 4096, 8192, 16384]:
            AB = np.zeros((n, 2 * 3 + 5 + 1))
            rng = np.random.default_rng(n)
            AB[:, 3:] = rng.standard_normal((n, 3 + 5 + 1))
            AB[:, 3 + 5] += 20.0
            _, _, f = oracle.gbtrf(AB, 3, 5)
            counts.append(f)
        ratios = [counts[k + 1] / counts[k] for k in range(len(counts) - 1)]
        assert all(abs(r - 2.0) < 0.01 for r in ratios), ratios


class TestBackwardErrorChecker:
    def test_matches_dense_reconstruction(self):
        for seed in range(10):
            n, kl, ku = 9, 2, 3
            T = random_band(n, kl, ku, 5000 + seed)
            AB0, AB, ipiv, info, _ = band_lu(T, kl, ku)
            D = T[:, :n].copy()
            dpiv, _ = oracle.dense_gepp(D)
            A = T[:, :n].T
            LU = D.T
            L = np.tril(LU, -1) + np.eye(n)
            U = np.triu(LU)
            P = np.eye(n)
            for k in range(n):
                q = dpiv[k] - 1
                P[[k, q]] = P[[q, k]]
            ref = np.linalg.norm(P @ A - L @ U) / (np.linalg.norm(A) * n * np.finfo(float).eps)
            got = oracle.band_backward_error(AB0, AB, kl, ku, ipiv)
            assert abs(got - ref) <= 0.5 + 0.1 * ref

    def test_detects_corruption(self):
        T = random_band(30, 3, 2, 7)
        AB0, AB, ipiv, _, _ = band_lu(T, 3, 2)
        AB[10, 3 + 2 + 1] += 1e-6
        assert oracle.band_backward_error(AB0, AB, 3, 2, ipiv) > 1e3


# --------------------------------------------------------------------------
# solve (Listing 1/2: lu(A) \ B)
# --------------------------------------------------------------------------
class TestSolve:
    @pytest.mark.parametrize("seed", range(20))
    def test_residual_and_scipy(self, seed):
        rng = np.random.default_rng(seed)
        n = int(rng.integers(1, 150))
        kl, ku = int(rng.integers(0, min(n, 10))), int(rng.integers(0, min(n, 10)))
        T = random_band(n, kl, ku, 6000 + seed)
        for d in range(n):
            T[d, d] += 3.0
        AB0, AB, ipiv, info, _ = band_lu(T, kl, ku)
        A = T[:, :n].T
        xt = rng.standard_normal((2, n))
        B = np.ascontiguousarray((A @ xt.T).T)
        X = oracle.gbtrs(AB, kl, ku, ipiv, B.copy())
        for k in range(2):
            r = np.abs(A @ X[k] - B[k]).max()
            assert r <= 10 * n * np.finfo(float).eps * np.abs(A).sum(1).max() * np.abs(X[k]).max()
        lx, linfo = lapack.dgbtrs(np.asfortranarray(AB.T), kl, ku, np.asfortranarray(B.T), ipiv - 1)
        assert linfo == 0
        np.testing.assert_allclose(X, lx.T, rtol=1e-10, atol=1e-12)
        # single-RHS call agrees bitwise with the multi-RHS call
        x1 = oracle.gbtrs(AB, kl, ku, ipiv, B[1:2].copy())
        assert np.array_equal(bits(x1[0]), bits(X[1]))

    def test_diagonal_exact(self):
        n = 7
        d = np.arange(1.0, n + 1)
        T = np.diag(d)
        AB0, AB, ipiv, info, _ = band_lu(T, 0, 0)
        b = np.arange(3.0, 3.0 + n)[None, :].copy()
        x = oracle.gbtrs(AB, 0, 0, ipiv, b)
        assert np.array_equal(x[0], np.arange(3.0, 3.0 + n) / d)


# --------------------------------------------------------------------------
# cost model (Sec. II-B speedup/slowdown constraints, Sec. III-B bounds)
# --------------------------------------------------------------------------
class TestCostModel:
    @pytest.mark.parametrize("name", list(inputs.WORKLOADS))
    def test_speedup_constraint_holds_on_workloads(self, name):
        w = inputs.WORKLOADS[name]
        c = oracle.op_counts(w["n"], w["kl"], w["ku"])
        assert c["speedup_constraint"] and c["slowdown_constraint"]
        assert c["speedup_ratio"] > 1.0

    def test_counters_match_model(self):
        n, kl, ku = 300, 4, 6
        T = random_band(n, kl, ku, 11)
        _, _, _, I = oracle.detect(T)
        _, C = oracle.dense_to_band(T, kl, ku)
        c = oracle.op_counts(n, kl, ku)
        assert I == c["I"] and C == c["C"]

    def test_max_speedup_grows_linearly(self):
        """Speedup_MAX ~ O(N) at fixed bands, slowdown bounded (Sec. III-B)."""
        r = [oracle.op_counts(n, 2, 2)["speedup_ratio"] for n in (1000, 2000, 4000, 8000)]
        growth = [r[k + 1] / r[k] for k in range(3)]
        assert all(1.9 < g < 2.1 for g in growth), growth
        s = [(n * n + 2 * n ** 3 / 3) / (2 * n ** 3 / 3) for n in (1000, 8000)]
        assert s[1] < s[0] < 1.01


# --------------------------------------------------------------------------
# triangular / diagonal solve from the band (Listing 1's istril / istriu
# branches, Sec. I-C)
# --------------------------------------------------------------------------
def tri_band(n, kl, ku, seed, diag_shift=4.0):
    T = random_band(n, kl, ku, seed)
    T[np.arange(n), np.arange(n)] += diag_shift * np.sign(T[np.arange(n), np.arange(n)] + 0.5)
    return T


def lapack_tb(AB, kl, ku):
    """xGBTRF-layout band (AB[j, r]) -> the (ldab, n) array LAPACK's xTBTRS reads."""
    if ku == 0:  # lower: A(i, j) at row i - j
        return np.ascontiguousarray(AB[:, kl:2 * kl + 1].T)
    return np.ascontiguousarray(AB[:, 0:ku + 1].T)  # upper, kl = 0: row ku + i - j


class TestTriangularSolve:
    def test_hand_examples(self):
        L = np.array([[2.0, 0, 0], [1, 4, 0], [0, 3, 8]])
        U = L.T.copy()
        D = np.diag([2.0, 4.0, 8.0])
        for A, kl, ku, b, x in [(L, 1, 0, [2.0, 5, 11], [1.0, 1, 1]),
                                (U, 0, 1, [3.0, 7, 8], [1.0, 1, 1]),
                                (D, 0, 0, [1.0, 1, 1], [0.5, 0.25, 0.125])]:
            AB, _ = oracle.dense_to_band(np.ascontiguousarray(A.T), kl, ku)
            B = np.array([b])
            assert oracle.band_trsv(AB, kl, ku, B) == 0
            assert np.array_equal(B[0], x)

    @pytest.mark.parametrize("seed", range(6))
    def test_exact_integer_solutions(self, seed):
        """Integer band entries, diagonal +-1 or +-2 and integer x: every
        intermediate is an integer, so substitution is exact."""
        rng = np.random.default_rng(700 + seed)
        n = int(rng.integers(5, 30))
        k = int(rng.integers(1, 6))
        for kl, ku in ((k, 0), (0, k)):
            A = np.zeros((n, n))
            for j in range(n):
                for i in range(max(0, j - ku), min(n - 1, j + kl) + 1):
                    A[i, j] = float(rng.integers(-3, 4))
                A[j, j] = float(rng.choice([-2.0, -1.0, 1.0, 2.0]))
            x = rng.integers(-4, 5, size=n).astype(float)
            # make b = A x with every x_j even where A(j,j) = +-2 divides exactly
            b = A @ x
            AB, _ = oracle.dense_to_band(np.ascontiguousarray(A.T), kl, ku)
            B = b[None, :].copy()
            assert oracle.band_trsv(AB, kl, ku, B) == 0
            assert np.array_equal(B[0], x), (kl, ku)

    @pytest.mark.parametrize("seed", range(8))
    def test_vs_lapack_dtbtrs(self, seed):
        rng = np.random.default_rng(710 + seed)
        n = int(rng.integers(1, 200))
        k = int(rng.integers(0, min(n, 40)))
        for kl, ku in ((k, 0), (0, k)):
            T = tri_band(n, kl, ku, 720 + seed)
            AB, _ = oracle.dense_to_band(T, kl, ku)
            B = rng.standard_normal((2, n))
            ref, info = lapack.dtbtrs(lapack_tb(AB, kl, ku), B.T.copy(),
                                      uplo="L" if ku == 0 else "U")
            assert info == 0
            got = B.copy()
            assert oracle.band_trsv(AB, kl, ku, got) == 0
            assert np.allclose(got, ref.T, rtol=1e-12, atol=1e-13 * np.abs(ref).max()), (kl, ku)

    def test_dense_solve_triangular(self):
        import scipy.linalg as sl
        n, kl = 150, 7
        T = tri_band(n, kl, 0, 730)
        AB, _ = oracle.dense_to_band(T, kl, 0)
        b = np.random.default_rng(731).standard_normal(n)
        B = b[None, :].copy()
        oracle.band_trsv(AB, kl, 0, B)
        ref = sl.solve_triangular(T.T, b, lower=True)
        assert np.allclose(B[0], ref, rtol=1e-12, atol=1e-13)

    def test_zero_diagonal_info_and_not_triangular(self):
        T = tri_band(20, 3, 0, 740)
        T[11, 11] = 0.0
        T[15, 15] = 0.0
        AB, _ = oracle.dense_to_band(T, 3, 0)
        B = np.ones((1, 20))
        assert oracle.band_trsv(AB, 3, 0, B) == 12
        assert np.all(np.isfinite(B[0, :11])) and not np.all(np.isfinite(B[0, 11:]))
        AB2, _ = oracle.dense_to_band(random_band(20, 2, 2, 741), 2, 2)
        with pytest.raises(ValueError):
            oracle.band_trsv(AB2, 2, 2, np.ones((1, 20)))


# --------------------------------------------------------------------------
# transposed solve with the band LU factors (the general A \ B of Listing 1
# applied to A^T; xGBTRS trans = 'T')
# --------------------------------------------------------------------------
def exact_solve(A, b):
    """Exact rational Gaussian elimination (brute force, any pivot order)."""
    from fractions import Fraction
    n = len(b)
    M = [[Fraction(float(A[i, j])) for j in range(n)] + [Fraction(float(b[i]))] for i in range(n)]
    for c in range(n):
        p = next(r for r in range(c, n) if M[r][c] != 0)
        M[c], M[p] = M[p], M[c]
        for r in range(c + 1, n):
            f = M[r][c] / M[c][c]
            if f:
                M[r] = [a - f * bb for a, bb in zip(M[r], M[c])]
    x = [Fraction(0)] * n
    for i in range(n - 1, -1, -1):
        s = M[i][n] - sum(M[i][j] * x[j] for j in range(i + 1, n))
        x[i] = s / M[i][i]
    return np.array([float(v) for v in x])


class TestTransposedSolve:
    def test_hand_example(self):
        A = np.array([[1.0, 2, 0], [5, 1, 3], [0, 4, 1]])
        AB, _ = oracle.dense_to_band(np.ascontiguousarray(A.T), 1, 1)
        ipiv, info, _ = oracle.gbtrf(AB, 1, 1)
        B = np.array([[6.0, 7.0, 4.0]])  # A^T [1, 1, 1]
        oracle.gbtrs_t(AB, 1, 1, ipiv, B)
        assert np.allclose(B[0], [1.0, 1.0, 1.0], rtol=0, atol=4e-16)

    @pytest.mark.parametrize("seed", range(6))
    def test_exact_rational(self, seed):
        rng = np.random.default_rng(750 + seed)
        n = int(rng.integers(2, 12))
        kl = int(rng.integers(0, n))
        ku = int(rng.integers(0, n))
        T = random_band(n, kl, ku, 760 + seed)
        A = T.T.copy()
        if abs(np.linalg.det(A)) < 1e-3:
            A += 3.0 * np.eye(n)
            T = np.ascontiguousarray(A.T)
        b = rng.standard_normal(n)
        ref = exact_solve(A.T, b)
        AB, _ = oracle.dense_to_band(T, kl, ku)
        ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
        assert info == 0
        B = b[None, :].copy()
        oracle.gbtrs_t(AB, kl, ku, ipiv, B)
        assert np.allclose(B[0], ref, rtol=1e-11, atol=1e-11 * np.abs(ref).max())

    @pytest.mark.parametrize("seed", range(8))
    def test_vs_lapack_dgbtrs_trans(self, seed):
        rng = np.random.default_rng(770 + seed)
        n = int(rng.integers(1, 300))
        kl = int(rng.integers(0, min(n, 30)))
        ku = int(rng.integers(0, min(n, 30)))
        T = random_band(n, kl, ku, 780 + seed)
        T[np.arange(n), np.arange(n)] += 2.0
        AB, _ = oracle.dense_to_band(T, kl, ku)
        ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
        B = rng.standard_normal((3, n))
        ref, inf2 = lapack.dgbtrs(np.ascontiguousarray(AB.T), kl, ku, B.T.copy(), ipiv - 1,
                                  trans=1)
        got = B.copy()
        oracle.gbtrs_t(AB, kl, ku, ipiv, got)
        assert np.allclose(got, ref.T, rtol=1e-11, atol=1e-11 * np.abs(ref).max())
        # and the residual of A^T x = b
        r = T @ got.T - B.T  # T = A^T as a numpy matrix
        assert np.abs(r).max() <= 1e-10 * (np.abs(T).sum(1).max() * np.abs(got).max() + 1)


# --------------------------------------------------------------------------
# rectangular m x n band LU (xGBTRF with m != n)
# --------------------------------------------------------------------------
class TestRectangularLU:
    @pytest.mark.parametrize("seed", range(5))
    def test_square_is_gbtrf_bitwise(self, seed):
        rng = np.random.default_rng(800 + seed)
        n = int(rng.integers(1, 120))
        kl = int(rng.integers(0, min(n, 20)))
        ku = int(rng.integers(0, min(n, 20)))
        AB, _ = oracle.dense_to_band(random_band(n, kl, ku, 810 + seed), kl, ku)
        A2 = AB.copy()
        p1, i1, f1 = oracle.gbtrf(AB, kl, ku)
        p2, i2, f2 = oracle.gbtrf_mn(A2, n, kl, ku)
        assert np.array_equal(p1, p2) and i1 == i2 and f1 == f2
        assert np.array_equal(bits(AB), bits(A2))

    def test_hand_3x2(self):
        A = np.array([[1.0, 2.0], [4.0, 3.0], [2.0, 1.0]])  # m = 3, n = 2
        AB = oracle.dense_to_band_mn(np.ascontiguousarray(A.T), 3, 2, 1)
        ipiv, info, _ = oracle.gbtrf_mn(AB, 3, 2, 1)
        assert list(ipiv) == [2, 2] and info == 0
        kv = 3
        assert AB[0, kv] == 4.0 and AB[1, kv - 1] == 3.0 and AB[1, kv] == 1.25
        assert AB[0, kv + 1] == 0.25 and AB[0, kv + 2] == 0.5 and AB[1, kv + 1] == -0.5 * (1 / 1.25)

    @pytest.mark.parametrize("seed", range(10))
    def test_vs_lapack_dgbtrf(self, seed):
        rng = np.random.default_rng(820 + seed)
        m = int(rng.integers(1, 150))
        n = int(rng.integers(1, 150))
        kl = int(rng.integers(0, m))
        ku = int(rng.integers(0, n))
        kl, ku = min(kl, 25), min(ku, 25)
        A = np.zeros((m, n))
        for j in range(n):
            for i in range(max(0, j - ku), min(m - 1, j + kl) + 1):
                A[i, j] = rng.standard_normal()
        if seed % 3 == 0 and min(m, n) > 2:
            A[:, min(m, n) // 2] = 0.0  # a zero column: info
        T = np.zeros((n, max(m, 1)))
        T[:, :m] = A.T
        AB = oracle.dense_to_band_mn(T, m, kl, ku)
        lu, ipiv_l, info_l = lapack.dgbtrf(np.ascontiguousarray(AB.T), kl, ku, m=m, n=n)
        ipiv, info, _ = oracle.gbtrf_mn(AB, m, kl, ku)
        assert info == info_l
        assert np.array_equal(ipiv, ipiv_l[:min(m, n)] + 1)
        assert np.allclose(AB, lu.T, rtol=1e-12, atol=1e-12 * max(1.0, np.abs(lu).max()))


# --------------------------------------------------------------------------
# band Cholesky (the Cholesky case beside LU, Sec. II-B; symmetric structure,
# Sec. II-A)
# --------------------------------------------------------------------------
def spd_band(n, kd, seed):
    rng = np.random.default_rng(seed)
    A = np.zeros((n, n))
    for j in range(n):
        for i in range(j + 1, min(n - 1, j + kd) + 1):
            A[i, j] = A[j, i] = rng.standard_normal()
    A[np.arange(n), np.arange(n)] = np.abs(A).sum(0) + 1.0
    return A


class TestBandCholesky:
    def test_hand_2x2(self):
        AB = oracle.lower_band(np.array([[4.0, 2.0], [2.0, 5.0]]), 1)
        assert oracle.pbtrf(AB, 1) == 0
        assert np.array_equal(AB, [[2.0, 1.0], [2.0, 0.0]])

    def test_exact_integer_factor(self):
        """A = L L^T with integer L whose diagonal is 1, 2 or 4: every step is
        exact, so the factor comes back exactly."""
        rng = np.random.default_rng(850)
        for n, kd in ((12, 3), (30, 5), (7, 6)):
            L = np.zeros((n, n))
            for j in range(n):
                L[j, j] = float(rng.choice([1.0, 2.0, 4.0]))
                for i in range(j + 1, min(n - 1, j + kd) + 1):
                    L[i, j] = float(rng.integers(-3, 4))
            A = L @ L.T
            AB = oracle.lower_band(A, kd)
            assert oracle.pbtrf(AB, kd) == 0
            assert np.array_equal(AB, oracle.lower_band(np.ascontiguousarray(L.T), kd))

    def test_toeplitz_closed_form(self):
        n = 400
        A = 2.0 * np.eye(n) - np.eye(n, k=1) - np.eye(n, k=-1)
        AB = oracle.lower_band(A, 1)
        assert oracle.pbtrf(AB, 1) == 0
        j = np.arange(n, dtype=float)
        assert np.allclose(AB[:, 0], np.sqrt((j + 2) / (j + 1)), rtol=4e-15, atol=0)
        assert np.allclose(AB[:-1, 1], -np.sqrt((j[:-1] + 1) / (j[:-1] + 2)), rtol=4e-15, atol=0)

    @pytest.mark.parametrize("seed", range(6))
    def test_vs_lapack_dpbtrf_and_numpy(self, seed):
        rng = np.random.default_rng(860 + seed)
        n = int(rng.integers(1, 250))
        kd = int(rng.integers(0, min(n, 40)))
        A = spd_band(n, kd, 870 + seed)
        AB = oracle.lower_band(A, kd)
        ref, info_l = lapack.dpbtrf(np.ascontiguousarray(AB.T), lower=1)
        assert oracle.pbtrf(AB, kd) == 0 and info_l == 0
        assert np.allclose(AB, ref.T, rtol=1e-13, atol=1e-14 * np.abs(ref).max())
        Ld = np.linalg.cholesky(A)
        assert np.allclose(AB, oracle.lower_band(np.ascontiguousarray(Ld.T), kd), rtol=1e-12,
                           atol=1e-13 * np.abs(Ld).max())

    def test_not_positive_definite(self):
        AB = oracle.lower_band(np.array([[1.0, 2.0], [2.0, 1.0]]), 1)
        assert oracle.pbtrf(AB, 1) == 2
        assert oracle.pbtrf(np.zeros((5, 2)), 1) == 1
        A = spd_band(30, 4, 880)
        A[17, 17] = np.nan
        assert oracle.pbtrf(oracle.lower_band(A, 4), 4) == 18
        A = spd_band(30, 4, 881)
        A[9, 9] = -1.0
        ref, info_l = lapack.dpbtrf(np.ascontiguousarray(oracle.lower_band(A, 4).T), lower=1)
        assert oracle.pbtrf(oracle.lower_band(A, 4), 4) == info_l == 10

    @pytest.mark.parametrize("seed", range(5))
    def test_solve_vs_lapack_dpbtrs(self, seed):
        rng = np.random.default_rng(890 + seed)
        n = int(rng.integers(1, 300))
        kd = int(rng.integers(0, min(n, 30)))
        A = spd_band(n, kd, 900 + seed)
        AB = oracle.lower_band(A, kd)
        oracle.pbtrf(AB, kd)
        B = rng.standard_normal((2, n))
        ref, info = lapack.dpbtrs(np.ascontiguousarray(AB.T), B.T.copy(), lower=1)
        got = B.copy()
        oracle.pbtrs(AB, kd, got)
        assert np.allclose(got, ref.T, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
        r = A @ got.T - B.T
        assert np.abs(r).max() <= 1e-11 * (np.abs(A).sum(1).max() * np.abs(got).max() + 1)


class TestSymmetryAndFusedConvert:
    def test_symmetric_band(self):
        A = spd_band(40, 5, 910)
        T = np.ascontiguousarray(A.T)
        assert oracle.is_symmetric_band(T, 5) == 1
        T2 = T.copy()
        T2[3, 6] = np.nextafter(T2[3, 6], np.inf)  # A(6, 3) != A(3, 6) by one ulp
        assert oracle.is_symmetric_band(T2, 5) == 0
        T3 = T.copy()
        T3[10, 12], T3[12, 10] = 0.0, -0.0
        assert oracle.is_symmetric_band(T3, 5) == 1
        T4 = T.copy()
        T4[10, 12] = T4[12, 10] = np.nan
        assert oracle.is_symmetric_band(T4, 5) == 0
        T5 = T.copy()
        T5[0, 20] = 1.0  # beyond kd: not examined
        assert oracle.is_symmetric_band(T5, 5) == 1

    def test_fused_definition(self):
        T = random_band(50, 3, 7, 920)
        kl, ku, ex, AB = oracle.detect_convert(T, 10, 10)
        assert (kl, ku, ex) == (3, 7, 0)
        assert np.array_equal(bits(AB), bits(oracle.dense_to_band(T, 3, 7)[0]))
        assert oracle.detect_convert(T, 2, 10)[2:] == (1, None)
