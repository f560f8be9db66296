"""GPU parity: every step of the HIP path against the CPU oracle on the same
seeded inputs.  Bandwidths, band arrays, pivots and info must match bit for
bit; the unblocked kernels also reproduce the factors and solutions bit for
bit (the same operations in the same order), which is stricter than the
1e-10 relative tolerance the method is held to."""
import numpy as np
import pytest

import oracle
from checks import assert_backward_error, assert_factors_close
from paper_2608_22099_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_22099_amd import bandlu  # noqa: E402  (loads libbandlu.so)

DEV = "cuda:0"


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def bits(x):
    return np.ascontiguousarray(x).view(np.uint64)


def assert_bitwise(g, o, what, nan_payload=False):
    """Bitwise equality.  A NaN that arithmetic produced may carry any payload
    (IEEE 754 leaves it open, and x86 and gfx950 differ), so unless
    nan_payload is set, two NaNs in the same slot count as equal."""
    g = np.ascontiguousarray(g)
    o = np.ascontiguousarray(o)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    diff = bits(g) != bits(o)
    if not nan_payload:
        diff &= ~(np.isnan(g) & np.isnan(o))
    bad = np.nonzero(diff)
    assert bad[0].size == 0, f"{what}: {bad[0].size} mismatches, first at {tuple(b[0] for b in bad)}: gpu={g[tuple(b[0] for b in bad)]!r} oracle={o[tuple(b[0] for b in bad)]!r}"


def gpu_pipeline(T, kl, ku, ldab=None, variant=None):
    """dense -> band -> getrf on the GPU; returns numpy (AB0, ABf, ipiv, info)."""
    A = to_dev(T)
    AB = bandlu.dense_to_band(A, kl, ku, ldab=ldab)
    AB0 = AB.cpu().numpy()
    ipiv, info = bandlu.band_getrf(AB, kl, ku, variant=variant)
    torch.cuda.synchronize()
    return AB0, AB.cpu().numpy(), ipiv.cpu().numpy(), int(info.cpu()[0])


def oracle_pipeline(T, kl, ku, ldab=None):
    n = T.shape[0]
    ldab = ldab or 2 * kl + ku + 1
    AB = np.zeros((n, ldab))
    AB, _ = oracle.dense_to_band(T, kl, ku, ldab=ldab, AB=AB)
    AB0 = AB.copy()
    ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
    return AB0, AB, ipiv, info


# ------------------------------------------------------------------ detect --
@pytest.mark.parametrize("seed", range(24))
def test_detect_random(seed):
    T, _, _ = inputs.random_case(seed, n_max=300 if seed % 2 else 40, special=True,
                                 lda_pad=seed % 3)
    o = oracle.detect(T)
    g = bandlu.band_detect(to_dev(T)).cpu().numpy()
    assert tuple(g) == o[:3]


def test_detect_special_values():
    n = 70
    for (i, j, v) in [(69, 0, np.nan), (0, 69, np.inf), (5, 2, 5e-324), (3, 60, -0.0)]:
        T = np.zeros((n, n))
        T[j, i] = v
        o = oracle.detect(T)
        g = bandlu.band_detect(to_dev(T)).cpu().numpy()
        assert tuple(g) == o[:3], (i, j, v)
    T = np.zeros((0, 1))
    assert tuple(bandlu.band_detect(to_dev(T)).cpu().numpy()) == (0, 0, 0)


@pytest.mark.parametrize("n", [1, 2, 3, 127, 128, 129, 255, 1000, 1023, 1025])
def test_detect_odd_sizes_and_alignment(n):
    rng = np.random.default_rng(n)
    kl, ku = int(rng.integers(0, n)), int(rng.integers(0, n))
    T = inputs.banded_dense(n, kl, ku, 7 + n, check=False)
    for pad in (0, 1):
        TT = np.zeros((n, n + pad))
        TT[:, :n] = T
        assert tuple(bandlu.band_detect(to_dev(TT)).cpu().numpy()) == oracle.detect(TT)[:3]


def test_detect_caps():
    T = inputs.banded_dense(2048, 40, 7, 3)
    A = to_dev(T)
    # caps at or above the true bandwidths: exact answer, no early exit
    assert tuple(bandlu.band_detect(A, 40, 7).cpu().numpy()) == (40, 7, 0)
    assert tuple(bandlu.band_detect(A, 100, 100).cpu().numpy()) == (40, 7, 0)
    # caps below: exceeded, values are lower bounds with one above its cap
    for kc, uc in [(39, -1), (-1, 6), (10, 3)]:
        kl, ku, ex = bandlu.band_detect(A, kc, uc).cpu().numpy()
        assert ex == 1 and kl <= 40 and ku <= 7
        assert (kc >= 0 and kl > kc) or (uc >= 0 and ku > uc)


def test_detect_batched():
    batch, n = 37, 90
    T = np.zeros((batch, n, n))
    want = []
    for b in range(batch):
        rng = np.random.default_rng(b)
        kl, ku = int(rng.integers(0, 12)), int(rng.integers(0, 12))
        inputs.banded_dense(n, kl, ku, 100 + b, out=T[b], check=False)
        want.append(oracle.detect(T[b])[:3])
    out, dmax = bandlu.band_detect_batched(to_dev(T))
    assert [tuple(r) for r in out.cpu().numpy()] == want
    w = np.array(want)
    assert tuple(dmax.cpu().numpy()) == (w[:, 0].max(), w[:, 1].max(), w[:, 2].max())
    out, dmax = bandlu.band_detect_batched(to_dev(T), 5, -1)
    o = out.cpu().numpy()
    for b in range(batch):
        assert o[b, 2] == int(want[b][0] > 5)
        if o[b, 2] == 0:
            assert tuple(o[b]) == want[b]


# ----------------------------------------------------------------- convert --
@pytest.mark.parametrize("seed", range(20))
def test_convert_random(seed):
    T, kl, ku = inputs.random_case(300 + seed, n_max=200, special=True, lda_pad=seed % 2)
    n = T.shape[0]
    ldab = 2 * kl + ku + 1 + seed % 3
    AB = torch.full((n, ldab), float("nan"), dtype=torch.float64, device=DEV)
    bandlu.dense_to_band(to_dev(T), kl, ku, AB=AB)
    o, _ = oracle.dense_to_band(T, kl, ku, ldab=ldab)
    assert_bitwise(AB.cpu().numpy(), o, "dense_to_band", nan_payload=True)


def test_convert_batched():
    batch, n, kl, ku = 50, 64, 5, 9
    T = np.stack([inputs.banded_dense(n, kl, ku, b) for b in range(batch)])
    AB = bandlu.dense_to_band_batched(to_dev(T), kl, ku).cpu().numpy()
    for b in range(batch):
        assert_bitwise(AB[b], oracle.dense_to_band(T[b], kl, ku)[0], f"batch {b}")


# ------------------------------------------------------------------- getrf --
def random_band(n, kl, ku, seed, shift=0.0):
    return inputs.banded_dense(n, kl, ku, seed, shift=shift, check=False)


@pytest.mark.parametrize("seed", range(40))
def test_getrf_random_shapes(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 200))
    kl = int(rng.integers(0, min(n, 40)))
    ku = int(rng.integers(0, min(n, 70)))
    T = random_band(n, kl, ku, 9000 + seed)
    g = gpu_pipeline(T, kl, ku)
    o = oracle_pipeline(T, kl, ku)
    variant = bandlu.band_getrf_variant(n, kl, ku)
    assert np.array_equal(g[2], o[2]), f"ipiv ({variant})"
    assert g[3] == o[3]
    what = f"factors ({variant}, n={n}, kl={kl}, ku={ku})"
    if variant in ("blocked_mfma", "wide"):
        assert_factors_close(g[1], o[1], kl, ku, what)
        assert_backward_error(o[0], g[1], kl, ku, g[2], what)
    else:
        assert_bitwise(g[1], o[1], what)


@pytest.mark.parametrize("kl,ku", [(0, 0), (1, 0), (0, 1), (3, 3), (16, 16), (2, 64), (31, 3),
                                   (23, 80), (8, 50), (5, 60), (24, 2)])
def test_getrf_window_boundaries(kl, ku):
    for n in (kl + ku + 1, 300):
        n = max(n, max(kl, ku) + 1)
        T = random_band(n, kl, ku, 77 + kl * 100 + ku)
        g = gpu_pipeline(T, kl, ku)
        o = oracle_pipeline(T, kl, ku)
        assert np.array_equal(g[2], o[2]) and g[3] == o[3]
        assert_bitwise(g[1], o[1], f"n={n} kl={kl} ku={ku}")


# The two-wavefront kernel and the one-wavefront window run the same
# operations: both must reproduce the oracle bit for bit, with and without
# row interchanges (no diagonal shift: interchanges at most steps).
SPLIT_SHAPES = [(2, 1, 0), (2, 1, 1), (3, 2, 0), (40, 1, 0), (50, 3, 2), (300, 3, 3), (300, 16, 16),
                (257, 31, 1), (65, 30, 3), (200, 2, 64), (300, 15, 97), (130, 8, 50), (1000, 5, 5),
                (129, 7, 0), (64, 1, 62)]


@pytest.mark.parametrize("n,kl,ku", SPLIT_SHAPES)
def test_getrf_split_exact(n, kl, ku):
    for shift in (0.0, float(kl + ku)):
        T = random_band(n, kl, ku, 31 + n + kl, shift=shift)
        o = oracle_pipeline(T, kl, ku)
        for variant in ("split", "window"):
            g = gpu_pipeline(T, kl, ku, variant=variant)
            what = f"{variant} n={n} kl={kl} ku={ku} shift={shift}"
            assert np.array_equal(g[2], o[2]), what
            assert g[3] == o[3], what
            assert_bitwise(g[1], o[1], what)


def test_getrf_split_special():
    """Singular columns, NaN entries, pivots below DBL_MIN and a zero matrix
    through the two-wavefront kernel."""
    n, kl, ku = 60, 3, 2
    cases = []
    for k in (0, 7, 59):
        T = random_band(n, kl, ku, 5 + k)
        T[k, :] = 0.0
        cases.append(("singular", T, kl, ku))
    T = random_band(n, kl, ku, 99)
    T[4, 4] = np.nan
    T[10, 12] = np.nan
    cases.append(("nan", T, kl, ku))
    cases.append(("tiny", random_band(n, 2, 2, 5) * 1e-300, 2, 2))
    cases.append(("zero", np.zeros((20, 20)), 2, 3))
    for what, T, a, c in cases:
        g = gpu_pipeline(T, a, c, variant="split")
        o = oracle_pipeline(T, a, c)
        assert np.array_equal(g[2], o[2]) and g[3] == o[3], what
        assert_bitwise(g[1], o[1], what)


# The one-wavefront window for kl <= 7 decides each pivot on scalars and runs
# blocks of 16 steps away from both ends without range tests: long bands that
# cross many 64-column periods (two columns per lane from 2kl+ku+1 = 65 on),
# lengths off the block size, and both widths at their limits.
LEAN_SHAPES = [(600, 0, 5), (601, 1, 1), (555, 2, 64), (700, 3, 3), (640, 4, 40), (603, 5, 100),
               (650, 6, 50), (700, 7, 20), (700, 7, 113), (700, 1, 61), (700, 1, 62), (97, 7, 6)]


@pytest.mark.parametrize("n,kl,ku", LEAN_SHAPES)
def test_getrf_window_lean_exact(n, kl, ku):
    for shift in (0.0, float(kl + ku)):
        T = random_band(n, kl, ku, 7 + n + 10 * kl + ku, shift=shift)
        check_exact(T, kl, ku, f"window n={n} kl={kl} ku={ku} shift={shift}", variant="window")


@pytest.mark.parametrize("kl,ku", [(3, 10), (2, 64), (7, 113)])
def test_getrf_window_lean_special(kl, ku):
    """Zero pivots, NaN and Inf entries, -0.0, and a column of subnormal
    numbers (its pivot is below DBL_MIN: the entries are divided) in the
    middle of the band, where the blocks take the lean steps."""
    n = 640
    T = random_band(n, kl, ku, 1234 + kl)
    T[:, 300] = 0.0                        # singular: info = 301 unless an earlier one
    T[:, 200] = 0.0
    T[320, max(0, 320 - min(kl, 1))] = np.nan
    T[400, 400 + min(ku, 1)] = np.inf
    T[450 - min(ku, 2): 451 + kl, 450] *= 1e-310   # subnormal column
    T[500, 500] = -0.0
    T[501, 501 + min(ku, 3)] = -0.0
    check_exact(T, kl, ku, f"special kl={kl} ku={ku}", variant="window")
    # a zero matrix and a matrix whose only nonzeros are tiny
    check_exact(np.zeros((n, n)), kl, ku, "zero", variant="window")
    check_exact(random_band(n, kl, ku, 99) * 1e-305, kl, ku, "tiny", variant="window")


def gbsv_lean_case(T, kl, ku, seed):
    """band_gbsv_lu + band_gbsv_back with one right-hand side (the lean
    window kernel runs the forward solve in its own steps) against the
    oracle's gbtrf + gbtrs, and against band_getrf + band_getrs."""
    n = T.shape[0]
    b = np.random.default_rng(seed).standard_normal((1, n))
    A = to_dev(T)
    AB1 = bandlu.dense_to_band(A, kl, ku)
    AB2 = AB1.clone()
    B1, B2 = to_dev(b), to_dev(b)
    ip1, inf1 = bandlu.band_getrf(AB1, kl, ku)
    bandlu.band_getrs(AB1, kl, ku, ip1, B1)
    ip2, inf2 = bandlu.band_gbsv_lu(AB2, kl, ku, B2)
    bandlu.band_gbsv_back(AB2, kl, ku, B2)
    torch.cuda.synchronize()
    ABo, _ = oracle.dense_to_band(T, kl, ku)
    ipo, info_o, _ = oracle.gbtrf(ABo, kl, ku)
    xo = b.copy()
    oracle.gbtrs(ABo, kl, ku, ipo, xo)
    what = f"gbsv n={n} kl={kl} ku={ku}"
    assert np.array_equal(ip2.cpu().numpy(), ipo) and int(inf2.cpu()[0]) == info_o, what
    assert_bitwise(AB2.cpu().numpy(), ABo, what + ": factors")
    assert_bitwise(B2.cpu().numpy(), xo, what + ": solution")
    assert torch.equal(ip1, ip2) and torch.equal(inf1, inf2)
    assert_bitwise(B2.cpu().numpy(), B1.cpu().numpy(), what + ": fused vs two calls")


@pytest.mark.parametrize("n,kl,ku", [(601, 1, 40), (555, 2, 64), (700, 3, 30), (640, 4, 40),
                                     (603, 5, 100), (650, 6, 50), (700, 6, 115), (33, 2, 30),
                                     (30, 1, 29), (40, 6, 30), (97, 3, 25)])
def test_gbsv_lean_fused(n, kl, ku):
    print(f"gbsv lean n={n} kl={kl} ku={ku}", flush=True)
    assert bandlu.band_getrf_variant(n, kl, ku) == "window"
    for shift in (0.0, float(kl + ku)):
        T = random_band(n, kl, ku, 4242 + n + kl, shift=shift)
        gbsv_lean_case(T, kl, ku, 17 + n)


@pytest.mark.parametrize("kl,ku", [(2, 64), (5, 30)])
def test_gbsv_lean_fused_special(kl, ku):
    """A zero column (its multipliers stay unscaled and enter the forward
    solve as stored), NaN and Inf entries and a subnormal pivot column."""
    n = 640
    T = random_band(n, kl, ku, 777 + kl)
    T[:, 300] = 0.0
    T[320, 320] = np.nan
    T[400, 400 + min(ku, 1)] = np.inf
    T[450 - min(ku, 2): 451 + kl, 450] *= 1e-310
    gbsv_lean_case(T, kl, ku, 99)
    T = random_band(n, kl, ku, 778 + kl)
    T[450 - min(ku, 2): 451 + kl, 450] *= 1e-310
    gbsv_lean_case(T, kl, ku, 98)


@pytest.mark.parametrize("seed", range(30))
def test_lean_window_random(seed):
    """Random shapes for the lean window kernel (kl <= 7, up to two columns
    per lane), forced, with zeros, NaN and tiny entries planted at random,
    and the fused forward solve where band_gbsv_lu takes it."""
    rng = np.random.default_rng(5000 + seed)
    kl = int(rng.integers(1, 8))
    ku = int(rng.integers(0, 128 - 2 * kl))
    n = int(rng.integers(max(kl, ku) + 1, 420))
    T = random_band(n, kl, ku, 6000 + seed, shift=float(rng.choice([0.0, 0.0, kl + ku])))
    for _ in range(int(rng.integers(0, 4))):
        i = int(rng.integers(0, n))
        j = int(rng.integers(max(0, i - kl), min(n, i + ku + 1)))
        T[i, j] = rng.choice([0.0, -0.0, np.nan, 1e-310, np.inf])
    if seed % 5 == 0:
        T[:, int(rng.integers(0, n))] = 0.0
    check_exact(T, kl, ku, f"lean random n={n} kl={kl} ku={ku}", variant="window")
    if kl <= 6 and bandlu.band_getrf_variant(n, kl, ku) == "window":
        gbsv_lean_case(T, kl, ku, 7000 + seed)


# The diagonal-pivot kernel must give the oracle's factors bit for bit
# whether every column keeps its diagonal pivot (dominant bands), a column
# fails the check (the two-wavefront kernel takes over there) or the first
# one does (no diagonal shift: interchanges at most steps).
DIAG_SHAPES = [(2, 1, 1), (3, 1, 1), (40, 1, 1), (300, 16, 16), (1000, 3, 3), (257, 1, 2),
               (129, 5, 8), (200, 11, 20), (97, 18, 16), (70, 1, 24), (64, 2, 9), (66, 7, 13),
               (500, 31, 1), (131, 9, 4), (77, 9, 17), (150, 6, 5), (90, 10, 15), (150, 23, 17),
               (100, 14, 24)]


def dominant_band(n, kl, ku, seed):
    return random_band(n, kl, ku, seed, shift=4.0 * (kl + ku + 1))


def check_exact(T, kl, ku, what, variant=None):
    g, o = gpu_pipeline(T, kl, ku, variant=variant), oracle_pipeline(T, kl, ku)
    assert np.array_equal(g[2], o[2]), f"{what}: ipiv"
    assert g[3] == o[3], f"{what}: info {g[3]} vs {o[3]}"
    assert_bitwise(g[1], o[1], what)
    return g, o


@pytest.mark.parametrize("n,kl,ku", DIAG_SHAPES)
def test_getrf_diag_exact(n, kl, ku):
    # (the default for 1 <= kl <= 4, 2kl+ku+1 <= 16 is WINDOW_G16: the
    # diagonal-pivot kernel is forced here, and the default checked too)
    assert bandlu.band_getrf_variant(n, kl, ku) == (
        "window_g16" if 1 <= kl <= 4 and 2 * kl + ku + 1 <= 16 else "diag")
    g, o = check_exact(dominant_band(n, kl, ku, 77 + n + ku), kl, ku, f"dominant n={n} kl={kl} ku={ku}",
                       variant="diag")
    assert np.array_equal(o[2], np.arange(1, n + 1))
    check_exact(random_band(n, kl, ku, 78 + n + ku), kl, ku, f"random n={n} kl={kl} ku={ku}",
                variant="diag")
    check_exact(random_band(n, kl, ku, 79 + n + ku), kl, ku, f"default kernel n={n} kl={kl} ku={ku}")


@pytest.mark.parametrize("n,kl,ku,cols", [(300, 16, 16, (0, 1, 2, 3, 17, 18, 19, 35, 36, 37, 53, 54, 100, 298, 299)),
                                          (129, 5, 8, (19, 20, 39, 40, 58, 59, 60, 61, 127, 128)),
                                          (90, 10, 15, (16, 17, 33, 88)),
                                          (2000, 16, 16, (71, 72, 73, 107, 500, 1000, 1511, 1998))])
def test_getrf_diag_resume(n, kl, ku, cols):
    """A dominant band with one weak diagonal: the diagonal-pivot kernel stops
    at that column (the last one has no candidates and never stops) and the
    two-wavefront kernel factors the rest."""
    for col in cols:
        T = dominant_band(n, kl, ku, 900 + col)
        T[col, col] = 1e-3  # T[j, i] is A[i, j]
        g, o = check_exact(T, kl, ku, f"weak diagonal {col} n={n} kl={kl} ku={ku}")
        assert (o[2][col] != col + 1) == (col < n - 1)
        assert np.array_equal(o[2][:col], np.arange(1, col + 1))


def test_getrf_diag_special():
    """Zero columns (info, no interchange), NaN on and below the diagonal,
    ties, pivots at and below DBL_MIN, a zero matrix and a zero column before
    a failing one, all through the diagonal-pivot kernel."""
    n, kl, ku = 120, 6, 5
    cases = []
    for k in (0, 7, 59, 119):
        T = dominant_band(n, kl, ku, 5 + k)
        T[k, :] = 0.0
        cases.append((f"zero column {k}", T))
    T = dominant_band(n, kl, ku, 99)
    T[4, 4] = np.nan    # NaN pivot: kept, as partial pivoting keeps it
    cases.append(("nan diagonal", T))
    T = dominant_band(n, kl, ku, 98)
    T[10, 12] = np.nan  # NaN candidate: never outranks the diagonal
    cases.append(("nan below", T))
    T = dominant_band(n, kl, ku, 97)
    T[0, 1] = -T[0, 0]  # |candidate| = |diagonal|: the diagonal wins the tie
    T[0, 3] = T[0, 0]
    cases.append(("ties", T))
    cases.append(("small", dominant_band(n, kl, ku, 96) * 1e-300))
    cases.append(("subnormal", dominant_band(n, kl, ku, 95) * 1e-310))
    cases.append(("zero matrix", np.zeros((n, n))))
    T = dominant_band(n, kl, ku, 94)
    T[20, :] = 0.0
    T[50, 50] = 1e-6
    cases.append(("zero column, then a failing one", T))
    for what, T in cases:
        g, o = check_exact(T, kl, ku, what, variant="diag")
        if what.split()[-1].isdigit():
            assert o[3] == int(what.split()[-1]) + 1
    g, o = check_exact(cases[-1][1], kl, ku, "info across the hand-over", variant="diag")
    assert o[3] == 21
    # long bands: a zero column and tiny pivots inside a chunk away from both
    # ends (the chunk is undone and replayed step by step)
    for col in (500, 719):
        T = dominant_band(2000, 16, 16, 70 + col)
        T[col, :] = 0.0
        g, o = check_exact(T, 16, 16, f"zero column {col}, n=2000", variant="diag")
        assert o[3] == col + 1
    T = dominant_band(2000, 16, 16, 71) * 1e-310
    check_exact(T, 16, 16, "subnormal pivots, n=2000", variant="diag")


def _column_scales(n):
    """Powers of ten from 1e-300 to 1e300 (and a subnormal scale) by column."""
    e = np.array([-300, -150, -20, 0, 20, 150, 300, -306, -310])
    return 10.0 ** np.tile(e, n // e.size + 1)[:n]


def test_getrf_diag_extreme_magnitudes():
    """Columns scaled from 1e-310 to 1e300 (pivot choices unchanged, pivots
    and their reciprocals across the exponent range, subnormal pivots that
    divide instead), through the diagonal-pivot kernel, bitwise."""
    for n, kl, ku in ((400, 16, 16), (300, 3, 3), (250, 7, 24)):
        T = dominant_band(n, kl, ku, 4242 + ku) * _column_scales(n)[:, None]  # row j of T is column j of A
        check_exact(T, kl, ku, f"scaled columns n={n} kl={kl} ku={ku}", variant="diag")
        check_exact(T, kl, ku, f"scaled columns, default kernel n={n} kl={kl} ku={ku}")


def test_getrf_diag_fill_rows_not_read():
    """Fill slots hold garbage on entry; both kernels of the variant write
    them (zeros, or fill-in after the hand-over)."""
    n, kl, ku = 200, 8, 6
    for weak in (None, 90):
        T = dominant_band(n, kl, ku, 8)
        if weak is not None:
            T[weak, weak] = 1e-4
        AB = bandlu.dense_to_band(to_dev(T), kl, ku)
        AB[:, :kl] = float("nan")
        ipiv, info = bandlu.band_getrf(AB, kl, ku, variant="diag")
        o = oracle_pipeline(T, kl, ku)
        got = AB.cpu().numpy()
        kv = kl + ku
        for j in range(n):  # slots outside the matrix keep what they held
            for r in range(kl):
                if r - kv + j < 0:
                    got[j, r] = 0.0
        assert np.array_equal(ipiv.cpu().numpy(), o[2]), weak
        assert_bitwise(got, o[1], f"fill rows, weak diagonal {weak}")


def test_getrf_diag_batched():
    """Each matrix of a batch stops (or not) on its own."""
    batch, n, kl, ku = 7, 180, 9, 11
    Ts = []
    for b in range(batch):
        T = dominant_band(n, kl, ku, 700 + b) if b % 3 != 2 else random_band(n, kl, ku, 700 + b)
        if b == 1:
            T[77, 77] = 1e-5
        if b == 4:
            T[30, :] = 0.0
        Ts.append(T)
    T = np.stack(Ts)
    AB = bandlu.dense_to_band_batched(to_dev(T), kl, ku)
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku)
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_bitwise(ABg[b], o[1], f"batch {b}")


def test_getrf_singular_and_nan():
    n, kl, ku = 50, 3, 2
    for k in [0, 7, 49]:
        T = random_band(n, kl, ku, 5 + k)
        T[k, :] = 0.0
        g, o = gpu_pipeline(T, kl, ku), oracle_pipeline(T, kl, ku)
        assert g[3] == o[3] == k + 1
        assert np.array_equal(g[2], o[2])
        assert_bitwise(g[1], o[1], "singular")
    T = random_band(n, kl, ku, 99)
    T[4, 4] = np.nan   # NaN on the diagonal: taken when first
    T[10, 12] = np.nan  # NaN below the diagonal: never taken
    g, o = gpu_pipeline(T, kl, ku), oracle_pipeline(T, kl, ku)
    assert np.array_equal(g[2], o[2]) and g[3] == o[3]
    assert_bitwise(g[1], o[1], "nan")
    Z = np.zeros((20, 20))
    g, o = gpu_pipeline(Z, 2, 3), oracle_pipeline(Z, 2, 3)
    assert g[3] == 1 and np.array_equal(g[2], o[2])
    assert_bitwise(g[1], o[1], "zero matrix")


def test_getrf_tiny_pivots():
    """|pivot| < DBL_MIN takes the division branch on both sides."""
    n, kl, ku = 40, 2, 2
    T = random_band(n, kl, ku, 5) * 1e-300
    g, o = gpu_pipeline(T, kl, ku), oracle_pipeline(T, kl, ku)
    assert np.array_equal(g[2], o[2])
    assert_bitwise(g[1], o[1], "tiny")


def test_getrf_fill_rows_not_read():
    n, kl, ku = 100, 4, 3
    T = random_band(n, kl, ku, 8)
    A = to_dev(T)
    AB = bandlu.dense_to_band(A, kl, ku)
    AB[:, :kl] = float("nan")
    ipiv, info = bandlu.band_getrf(AB, kl, ku)
    o = oracle_pipeline(T, kl, ku)
    got = AB.cpu().numpy()
    kv = kl + ku
    for j in range(n):  # slots outside the matrix keep what they held
        for r in range(kl):
            if r - kv + j < 0:
                got[j, r] = 0.0
    assert np.array_equal(ipiv.cpu().numpy(), o[2])
    assert_bitwise(got, o[1], "fill rows")


@pytest.mark.parametrize("kl,ku,batch,n", [(4, 4, 256, 64), (1, 2, 100, 33), (7, 3, 70, 50),
                                           (4, 4, 3, 64), (10, 5, 65, 40), (3, 20, 64, 90),
                                           (3, 30, 5, 300), (2, 64, 7, 200), (6, 40, 63, 120)])
def test_getrf_batched(kl, ku, batch, n):
    # (the last three: batches below 64 beyond the sixteen-lane and diagonal
    # kernels, which the lean window kernel factors one matrix per workgroup)
    T = np.stack([random_band(n, kl, ku, 500 + b) for b in range(batch)])
    T[1 % batch, 3, :] = 0.0  # one singular matrix
    A = to_dev(T)
    AB = bandlu.dense_to_band_batched(A, kl, ku)
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku)
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_bitwise(ABg[b], o[1], f"batch {b}")


def test_getrf_deterministic():
    T = random_band(3000, 16, 16, 1)
    a = gpu_pipeline(T, 16, 16)
    b = gpu_pipeline(T, 16, 16)
    assert_bitwise(a[1], b[1], "rerun")


# ------------------------------------------------------------------- getrs --
@pytest.mark.parametrize("seed", range(16))
def test_getrs_random(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    kl = int(rng.integers(0, min(n, 30)))
    ku = int(rng.integers(0, min(n, 90)))
    nrhs = int(rng.integers(1, 4))
    T = random_band(n, kl, ku, 700 + seed, shift=4.0)
    _, ABo, ipo, _ = oracle_pipeline(T, kl, ku)
    B = rng.standard_normal((nrhs, n))
    xo = oracle.gbtrs(ABo, kl, ku, ipo, B.copy())
    Bg = to_dev(B)
    bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg)
    assert_bitwise(Bg.cpu().numpy(), xo, f"getrs n={n} kl={kl} ku={ku}")


def test_getrs_large_bands():
    for n, kl, ku in [(700, 70, 100), (2000, 200, 300)]:
        T = random_band(n, kl, ku, n, shift=float(kl + ku))
        _, ABo, ipo, _ = oracle_pipeline(T, kl, ku)
        B = np.random.default_rng(n).standard_normal((1, n))
        xo = oracle.gbtrs(ABo, kl, ku, ipo, B.copy())
        Bg = to_dev(B)
        bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg)
        assert_bitwise(Bg.cpu().numpy(), xo, f"getrs n={n}")


def test_getrs_global_path():
    n, kl, ku = 9000, 3, 5  # right-hand side larger than the LDS path
    T = random_band(n, kl, ku, 4, shift=10.0)
    _, ABo, ipo, _ = oracle_pipeline(T, kl, ku)
    B = np.random.default_rng(1).standard_normal((2, n))
    xo = oracle.gbtrs(ABo, kl, ku, ipo, B.copy())
    Bg = to_dev(B)
    bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg)
    assert_bitwise(Bg.cpu().numpy(), xo, "getrs global")


def test_getrs_batched():
    batch, n, kl, ku, nrhs = 40, 80, 4, 4, 2
    T = np.stack([random_band(n, kl, ku, 900 + b) for b in range(batch)])
    outs = [oracle_pipeline(T[b], kl, ku) for b in range(batch)]
    AB = np.stack([o[1] for o in outs])
    ip = np.stack([o[2] for o in outs])
    B = np.random.default_rng(3).standard_normal((batch, nrhs, n))
    Bg = to_dev(B)
    bandlu.band_getrs_batched(to_dev(AB), kl, ku, to_dev(ip), Bg)
    got = Bg.cpu().numpy()
    for b in range(batch):
        xo = oracle.gbtrs(AB[b], kl, ku, ip[b], B[b].copy())
        assert_bitwise(got[b], xo, f"batch {b}")


# Every solve kernel computes the same operations in the same order: each
# must reproduce the oracle bit for bit wherever it applies.
SOLVE_SHAPES = [(1, 0, 0), (2, 1, 0), (2, 0, 1), (3, 1, 1), (65, 64, 0), (70, 3, 66), (129, 10, 60),
                (300, 63, 64), (500, 64, 63), (640, 127, 1), (700, 70, 100), (900, 128, 127),
                (1000, 3, 3), (1200, 200, 300), (1500, 255, 300), (2000, 300, 700), (3000, 16, 16)]


@pytest.mark.parametrize("n,kl,ku", SOLVE_SHAPES)
def test_getrs_ring_exact(n, kl, ku):
    rng = np.random.default_rng(n + 7 * kl + 13 * ku)
    nrhs = 1 + (n % 3)
    # pivoting inputs (no diagonal shift) as well as dominant ones
    T = random_band(n, kl, ku, 1100 + n + kl, shift=0.0 if n % 2 else float(kl + ku))
    _, ABo, ipo, _ = oracle_pipeline(T, kl, ku)
    B = rng.standard_normal((nrhs, n))
    xo = oracle.gbtrs(ABo, kl, ku, ipo, B.copy())
    Bg = to_dev(B)
    bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg, variant="ring")
    assert_bitwise(Bg.cpu().numpy(), xo, f"ring getrs n={n} kl={kl} ku={ku}")


@pytest.mark.parametrize("n,kl,ku", [(1000, 3, 3), (300, 40, 20), (129, 10, 53), (90, 63, 0)])
def test_getrs_window_exact(n, kl, ku):
    T = random_band(n, kl, ku, 1300 + n, shift=0.0)
    _, ABo, ipo, _ = oracle_pipeline(T, kl, ku)
    B = np.random.default_rng(n).standard_normal((2, n))
    xo = oracle.gbtrs(ABo, kl, ku, ipo, B.copy())
    for variant in ("window", "generic"):
        Bg = to_dev(B)
        bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg, variant=variant)
        assert_bitwise(Bg.cpu().numpy(), xo, f"{variant} getrs n={n} kl={kl} ku={ku}")


LANE_SHAPES = [(1, 0, 0), (2, 1, 0), (2, 0, 1), (3, 1, 1), (63, 5, 3), (64, 16, 16), (65, 16, 16),
               (66, 2, 7), (127, 20, 23), (128, 10, 43), (129, 1, 61), (200, 0, 20), (300, 16, 16),
               (1000, 3, 3), (8191, 16, 16), (641, 21, 21), (97, 0, 63)]


@pytest.mark.parametrize("n,kl,ku", LANE_SHAPES)
def test_getrs_lane_exact(n, kl, ku):
    """The lane-per-row solve, bitwise against the oracle, with interchanges
    (factors of a random band) and without (a dominant band), and with
    several right-hand sides."""
    for shift, nrhs in ((0.0, 1), (4.0 * (kl + ku + 1), 3)):
        T = random_band(n, kl, ku, 61 + n + kl + ku, shift=shift)
        ABo = oracle_pipeline(T, kl, ku)[1]
        ipo = oracle_pipeline(T, kl, ku)[2]
        B = np.random.default_rng(n + kl).standard_normal((nrhs, n))
        xo = B.copy()
        oracle.gbtrs(ABo, kl, ku, ipo, xo)
        Bg = to_dev(B)
        if nrhs == 1:
            assert bandlu.band_getrs_variant(n, kl, ku) == "lane"
        bandlu.band_getrs(to_dev(ABo), kl, ku, to_dev(ipo), Bg, variant="lane")
        assert_bitwise(Bg.cpu().numpy(), xo, f"lane getrs n={n} kl={kl} ku={ku} nrhs={nrhs}")


def test_getrs_lane_batched_and_special():
    """Batched systems through the lane solve; a right-hand side with a NaN,
    infinities and zeros."""
    batch, n, kl, ku = 5, 150, 6, 9
    T = np.stack([random_band(n, kl, ku, 800 + b, shift=(0.0 if b % 2 else 30.0)) for b in range(batch)])
    outs = [oracle_pipeline(T[b], kl, ku) for b in range(batch)]
    AB = np.stack([o[1] for o in outs])
    ip = np.stack([o[2] for o in outs]).astype(np.int32)
    B = np.random.default_rng(5).standard_normal((batch, 2, n))
    B[1, 0, 7] = np.nan
    B[2, 1, 100] = np.inf
    B[3, 0, :] = 0.0
    xo = B.copy()
    for b in range(batch):
        oracle.gbtrs(AB[b], kl, ku, ip[b], xo[b])
    Bg = to_dev(B)
    bandlu.band_getrs_batched(to_dev(AB), kl, ku, to_dev(ip), Bg, variant="lane")
    got = Bg.cpu().numpy()
    for b in range(batch):
        assert_bitwise(got[b], xo[b], f"batch {b}")


def test_getrs_lane_extreme_magnitudes():
    """The lane solve with a diagonal of U from 1e-310 to 1e300 and
    right-hand sides with tiny, huge and subnormal entries (the division's
    scaled cases), bitwise against the oracle."""
    for n, kl, ku in ((700, 16, 16), (500, 21, 21), (300, 2, 5)):
        T = dominant_band(n, kl, ku, 4343 + ku) * _column_scales(n)[:, None]
        o = oracle_pipeline(T, kl, ku)
        rng = np.random.default_rng(n + ku)
        B = rng.standard_normal((2, n)) * 10.0 ** rng.choice([-300, -200, 0, 200, 300], size=(2, n))
        B[0, ::13] = 5e-324
        xo = B.copy()
        oracle.gbtrs(o[1], kl, ku, o[2], xo)
        Bg = to_dev(B)
        assert bandlu.band_getrs_variant(n, kl, ku) == "lane"
        bandlu.band_getrs(to_dev(o[1]), kl, ku, to_dev(o[2]), Bg)
        assert_bitwise(Bg.cpu().numpy(), xo, f"scaled lane getrs n={n} kl={kl} ku={ku}")


def test_getrs_ring_batched_and_padded():
    batch, n, kl, ku, nrhs = 5, 400, 70, 90, 2
    T = np.stack([random_band(n, kl, ku, 1400 + b) for b in range(batch)])
    outs = [oracle_pipeline(T[b], kl, ku) for b in range(batch)]
    AB = np.stack([o[1] for o in outs])
    ip = np.stack([o[2] for o in outs])
    ldb = n + 5  # padded right-hand sides: rows n..ldb-1 must stay untouched
    B = np.random.default_rng(5).standard_normal((batch, nrhs, ldb))
    Bg = to_dev(B)
    bandlu.band_getrs_batched(to_dev(AB), kl, ku, to_dev(ip), Bg[:, :, :n], variant="ring")
    got = Bg.cpu().numpy()
    for b in range(batch):
        xo = oracle.gbtrs(AB[b], kl, ku, ip[b], B[b, :, :n].copy())
        assert_bitwise(got[b, :, :n], xo, f"batch {b}")
    assert_bitwise(got[:, :, n:], B[:, :, n:], "padding", nan_payload=True)


def test_getrs_ring_unsupported():
    n, kl, ku = 2000, 500, 600  # kl + ku > 1023
    AB = torch.zeros((n, 2 * kl + ku + 1), dtype=torch.float64, device=DEV)
    ip = torch.ones(n, dtype=torch.int32, device=DEV)
    with pytest.raises(bandlu.BandLUError):
        bandlu.band_getrs(AB, kl, ku, ip, torch.zeros((1, n), dtype=torch.float64, device=DEV),
                          variant="ring")
    assert bandlu.band_getrs_variant(32768, 256, 256) == "ring"
    assert bandlu.band_getrs_variant(256, 4, 4, 1, 4096) == "g16"


# ----------------------------------------------------------- blocked getrf --
BLOCKED_SHAPES = [(300, 40, 3), (95, 20, 52), (700, 100, 150), (1100, 256, 256), (530, 33, 200),
                  (64, 63, 63), (257, 32, 0), (400, 250, 1), (300, 31, 90), (97, 12, 80)]


@pytest.mark.parametrize("n,kl,ku", BLOCKED_SHAPES)
def test_getrf_blocked_exact(n, kl, ku):
    """The blocked kernel with rank-1 trailing updates is bitwise the unblocked
    algorithm (forced through band_getrf_ex where the matrix-core variant
    would be chosen)."""
    T = random_band(n, kl, ku, 31 * n + kl)
    g, o = gpu_pipeline(T, kl, ku, variant="blocked"), oracle_pipeline(T, kl, ku)
    assert np.array_equal(g[2], o[2]) and g[3] == o[3]
    assert_bitwise(g[1], o[1], f"blocked n={n} kl={kl} ku={ku}")


def test_getrf_blocked_batched_and_singular():
    batch, n, kl, ku = 5, 200, 40, 30
    T = np.stack([random_band(n, kl, ku, 70 + b) for b in range(batch)])
    T[2, 77, :] = 0.0
    AB = bandlu.dense_to_band_batched(to_dev(T), kl, ku)
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku, variant="blocked")
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_bitwise(ABg[b], o[1], f"batch {b}")


# ------------------------------------------------------ matrix-core getrf --
def check_mfma(T, kl, ku, what, variant=None):
    """The matrix-core kernels against the oracle: the default choice (the
    persistent kernel where the batch fits one launch) and, unless a variant
    is named, the one-launch-per-panel kernel as well."""
    o = oracle_pipeline(T, kl, ku)
    for v in ([variant] if variant else [None, "blocked_mfma"]):
        g = gpu_pipeline(T, kl, ku, variant=v)
        w = f"{what} ({v or bandlu.band_getrf_variant(T.shape[0], kl, ku)})"
        assert np.array_equal(g[2], o[2]), f"{w}: ipiv"
        assert g[3] == o[3], f"{w}: info {g[3]} vs {o[3]}"
        assert_factors_close(g[1], o[1], kl, ku, w)
        if np.any(o[0] != 0.0):
            assert_backward_error(o[0], g[1], kl, ku, g[2], w)
    return g, o


@pytest.mark.parametrize("n,kl,ku", [(300, 40, 3), (700, 100, 150), (1100, 256, 256), (530, 33, 200),
                                     (64, 63, 63), (257, 32, 0), (400, 250, 1), (33, 32, 0),
                                     (64, 32, 31), (65, 40, 24), (96, 50, 45), (289, 256, 32),
                                     (600, 256, 343), (128, 127, 0)])
def test_getrf_mfma_shapes(n, kl, ku):
    """Panels of 32 with a ragged last panel, bands that reach one or many
    column blocks, kl at both ends of the variant's range."""
    assert bandlu.band_getrf_variant(n, kl, ku) == "wide"
    check_mfma(random_band(n, kl, ku, 7 * n + kl + ku), kl, ku, f"n={n} kl={kl} ku={ku}")


@pytest.mark.parametrize("seed", range(12))
def test_getrf_mfma_random(seed):
    rng = np.random.default_rng(4000 + seed)
    n = int(rng.integers(33, 900))
    kl = int(rng.integers(32, min(n, 257)))
    ku = int(rng.integers(0, min(n, 300)))
    check_mfma(random_band(n, kl, ku, 600 + seed), kl, ku, f"seed {seed} n={n} kl={kl} ku={ku}")


@pytest.mark.parametrize("n,kl,ku", [(40, 0, 0), (70, 3, 2), (100, 10, 5), (50, 20, 49),
                                     (31, 5, 5), (1, 0, 0), (2, 1, 1)])
def test_getrf_mfma_forced_narrow(n, kl, ku):
    """The matrix-core kernels also factor narrow bands when forced (blocks
    narrower than a panel, a band that does not reach the next panel)."""
    for v in ("blocked_mfma", "wide"):
        check_mfma(random_band(n, kl, ku, 11 * n + kl), kl, ku, f"forced n={n} kl={kl} ku={ku}",
                   variant=v)


def test_getrf_mfma_pivoting_and_singular():
    """Heavy pivoting (rows scaled so the pivot is rarely the diagonal) and
    exactly singular columns: info and ipiv match; a zero column leaves the
    factorisation running."""
    n, kl, ku = 300, 40, 20
    T = random_band(n, kl, ku, 42)
    T *= np.exp(np.random.default_rng(1).uniform(-3, 3, size=(1, n)))  # scales rows of A
    check_mfma(T, kl, ku, "scaled rows")
    for col in (0, 31, 32, 200, n - 1):
        S = random_band(n, kl, ku, 43 + col)
        S[col, :] = 0.0  # T[j, :] is column j of A
        g, o = check_mfma(S, kl, ku, f"zero column {col}")
        assert o[3] == col + 1
    Z = np.zeros((70, 70))
    g, o = check_mfma(Z, 33, 2, "zero matrix")
    assert g[3] == 1


@pytest.mark.parametrize("n,kl,ku", [(300, 40, 3), (1100, 256, 256), (257, 32, 0), (65, 40, 24),
                                     (600, 256, 343), (97, 96, 5)])
def test_getrf_mfma_no_interchange(n, kl, ku):
    """Diagonally dominant bands: every panel keeps its diagonal pivots, so
    the kernel's no-interchange attempt passes on every panel."""
    T = random_band(n, kl, ku, 17 * n + kl, shift=4.0 * (kl + 1))
    g, o = check_mfma(T, kl, ku, f"dominant n={n} kl={kl} ku={ku}")
    assert np.array_equal(o[2], np.arange(1, n + 1))


@pytest.mark.parametrize("col", [0, 1, 30, 31, 32, 63, 64, 95, 190, 191])
def test_getrf_mfma_late_interchange(col):
    """A dominant band with one weak diagonal: the no-interchange attempt runs
    up to that column of its panel, then the panel is factored again with
    pivoting; panels before and after pass."""
    n, kl, ku = 192, 48, 20
    T = random_band(n, kl, ku, 900 + col, shift=4.0 * (kl + 1))
    T[col, col] = 1e-3  # T[j, i] is A[i, j]
    g, o = check_mfma(T, kl, ku, f"weak diagonal {col}")
    assert o[2][col] != col + 1 or col == n - 1


def test_getrf_mfma_no_interchange_ties_and_zeros():
    """Cases decided without an interchange: a candidate equal in magnitude
    to the diagonal (the diagonal wins the tie), and a zero column in a
    dominant band (zero pivot, info set, factorisation goes on)."""
    n, kl, ku = 200, 40, 10
    T = random_band(n, kl, ku, 77, shift=4.0 * (kl + 1))
    T[0, 1] = -T[0, 0]  # A[1, 0] = -A[0, 0]
    T[0, 5] = T[0, 0]
    g, o = check_mfma(T, kl, ku, "tie in the first column")
    assert o[2][0] == 1
    for col in (0, 33, 63, 199):
        S = random_band(n, kl, ku, 78 + col, shift=4.0 * (kl + 1))
        S[col, :] = 0.0
        g, o = check_mfma(S, kl, ku, f"zero column {col} in a dominant band")
        assert o[3] == col + 1


def test_getrf_mfma_no_interchange_batched():
    """A batch mixing dominant systems (no interchange) with ones that pivot."""
    batch, n, kl, ku = 5, 230, 48, 40
    T = np.stack([random_band(n, kl, ku, 310 + b, shift=(4.0 * (kl + 1) if b % 2 == 0 else 0.0))
                  for b in range(batch)])
    AB = bandlu.dense_to_band_batched(to_dev(T), kl, ku)
    AB0 = AB.cpu().numpy()
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku)
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_factors_close(ABg[b], o[1], kl, ku, f"batch {b}")
        assert_backward_error(AB0[b], ABg[b], kl, ku, ipg[b], f"batch {b}")


def test_getrf_mfma_batched():
    batch, n, kl, ku = 6, 230, 48, 40
    T = np.stack([random_band(n, kl, ku, 300 + b) for b in range(batch)])
    T[3, 100, :] = 0.0
    AB = bandlu.dense_to_band_batched(to_dev(T), kl, ku)
    AB0 = AB.cpu().numpy()
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku)
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_factors_close(ABg[b], o[1], kl, ku, f"batch {b}")
        assert_backward_error(AB0[b], ABg[b], kl, ku, ipg[b], f"batch {b}")


def test_getrf_mfma_deterministic():
    T = random_band(700, 64, 64, 3)
    a = gpu_pipeline(T, 64, 64)
    b = gpu_pipeline(T, 64, 64)
    assert_bitwise(a[1], b[1], "rerun")


# ---------------------------------------------------- one-workgroup getrf --
def special_band(n, kl, ku, seed, neg_zero=0.0, nans=0, zero_cols=()):
    """A random band with in-band -0.0 entries (fraction neg_zero), a few NaNs
    and zeroed columns: the inputs where only the exact update extent keeps a
    kernel bitwise equal to the unblocked algorithm."""
    T = random_band(n, kl, ku, seed)
    rng = np.random.default_rng(seed + 1)
    j, i = inputs.band_index(n, kl, ku)
    if neg_zero:
        pick = rng.random(j.size) < neg_zero
        T[j[pick], i[pick]] = -0.0
    for q in rng.choice(j.size, size=min(nans, j.size), replace=False) if nans else ():
        T[j[q], i[q]] = np.nan
    for c in zero_cols:
        T[c, :] = 0.0
    return T


@pytest.mark.parametrize("seed", range(16))
def test_getrf_generic_forced(seed):
    """The one-workgroup kernel (the default beyond kl = 256) forced on random
    shapes, with -0.0 entries, NaNs and singular columns: bitwise."""
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.integers(1, 160))
    kl, ku = int(rng.integers(0, n)), int(rng.integers(0, n))
    T = special_band(n, kl, ku, 7100 + seed, neg_zero=0.2 if seed % 2 else 0.0,
                     nans=seed % 3, zero_cols=(n // 2,) if seed % 4 == 1 else ())
    g = gpu_pipeline(T, kl, ku, variant="generic")
    o = oracle_pipeline(T, kl, ku)
    assert np.array_equal(g[2], o[2]) and g[3] == o[3]
    assert_bitwise(g[1], o[1], f"generic n={n} kl={kl} ku={ku}")


@pytest.mark.parametrize("n,kl,ku", [(600, 300, 20), (400, 399, 0), (700, 257, 257)])
def test_getrf_generic_default(n, kl, ku):
    """kl > 256 runs the one-workgroup kernel by default."""
    assert bandlu.band_getrf_variant(n, kl, ku) == "generic"
    for zero in (None, n // 3):
        T = special_band(n, kl, ku, 7300 + n, neg_zero=0.05, zero_cols=() if zero is None else (zero,))
        g, o = gpu_pipeline(T, kl, ku), oracle_pipeline(T, kl, ku)
        assert np.array_equal(g[2], o[2]) and g[3] == o[3]
        assert_bitwise(g[1], o[1], f"generic default n={n} kl={kl} ku={ku} zero col {zero}")


# A leading dimension above 2kl+ku+1 must neither change the result nor send
# the call to a slower kernel than needed (the choice falls back through the
# kernels that fit before the one-workgroup kernel).
@pytest.mark.parametrize("n,kl,ku,pad,shift", [(500, 3, 5, 1, 20.0), (500, 3, 5, 7, 0.0),
                                               (400, 16, 16, 1, 0.0), (300, 16, 16, 3, 40.0),
                                               (300, 0, 10, 2, 0.0), (300, 2, 64, 5, 0.0),
                                               (300, 20, 100, 4, 0.0), (200, 40, 30, 3, 0.0)])
def test_getrf_padded_ldab(n, kl, ku, pad, shift):
    ldab = 2 * kl + ku + 1 + pad
    T = random_band(n, kl, ku, 8100 + n + kl + pad, shift=shift)
    g = gpu_pipeline(T, kl, ku, ldab=ldab)
    o = oracle_pipeline(T, kl, ku, ldab=ldab)
    assert np.array_equal(g[2], o[2]) and g[3] == o[3]
    what = f"padded ldab={ldab} n={n} kl={kl} ku={ku}"
    if kl >= 32:
        assert_factors_close(g[1][:, :ldab - pad], o[1][:, :ldab - pad], kl, ku, what)
    else:
        assert_bitwise(g[1][:, :ldab - pad], o[1][:, :ldab - pad], what)
    # rows beyond 2kl+ku are never written
    assert_bitwise(g[1][:, ldab - pad:], g[0][:, ldab - pad:], what + " (padding rows)",
                   nan_payload=True)


def test_getrf_padded_ldab_batched():
    batch, n, kl, ku = 70, 64, 4, 4
    ldab = 2 * kl + ku + 1 + 3
    T = np.stack([random_band(n, kl, ku, 8200 + b) for b in range(batch)])
    AB = torch.zeros((batch, n, ldab), dtype=torch.float64, device=DEV)
    bandlu.dense_to_band_batched(to_dev(T), kl, ku, AB=AB)
    ipiv, info = bandlu.band_getrf_batched(AB, kl, ku)
    ABg, ipg, infg = AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy()
    for b in range(batch):
        o = oracle_pipeline(T[b], kl, ku, ldab=ldab)
        assert np.array_equal(ipg[b], o[2]) and infg[b] == o[3], b
        assert_bitwise(ABg[b], o[1], f"batch {b}")


@pytest.mark.parametrize("n,kl,ku", [(300, 20, 100), (200, 5, 120), (300, 40, 3), (500, 31, 90)])
def test_getrf_blocked_special_values(n, kl, ku):
    """The blocked kernel applies each step only up to the step's update
    extent and skips zero pivots, as the unblocked algorithm does, so in-band
    -0.0 entries, NaNs and zero columns come out bitwise the same."""
    for k, (nz, nans, zc) in enumerate([(0.3, 0, ()), (0.1, 2, ()), (0.2, 0, (n // 3, n // 3 + 1))]):
        T = special_band(n, kl, ku, 8300 + n + k, neg_zero=nz, nans=nans, zero_cols=zc)
        g = gpu_pipeline(T, kl, ku, variant="blocked")
        o = oracle_pipeline(T, kl, ku)
        assert np.array_equal(g[2], o[2]) and g[3] == o[3]
        assert_bitwise(g[1], o[1], f"blocked specials n={n} kl={kl} ku={ku} case {k}")


# ------------------------------------------------------ any-band solve --
@pytest.mark.parametrize("n,kl,ku,nrhs", [(1500, 600, 500, 2), (8300, 10, 1020, 1), (1100, 1000, 90, 1)])
def test_getrs_any_band(n, kl, ku, nrhs):
    """kl+ku+1 > 1024: the any-band solve, with the right-hand sides in LDS
    (n <= 8192) and in global memory, bitwise."""
    T = random_band(n, kl, ku, 8400 + n, shift=float(kl + ku))
    o = oracle_pipeline(T, kl, ku)
    B = np.random.default_rng(n).standard_normal((nrhs, n))
    Bg = to_dev(B)
    bandlu.band_getrs(to_dev(o[1]), kl, ku, to_dev(o[2]), Bg)
    xo = oracle.gbtrs(o[1], kl, ku, o[2], B.copy())
    assert_bitwise(Bg.cpu().numpy(), xo, f"any-band getrs n={n} kl={kl} ku={ku}")
    Bg = to_dev(B)
    bandlu.band_getrs(to_dev(o[1]), kl, ku, to_dev(o[2]), Bg, variant="generic")
    assert_bitwise(Bg.cpu().numpy(), xo, "forced generic")
