"""GPU parity for the branches beyond the LU path, against the CPU oracle, bit
for bit (every kernel here performs the oracle's operations in its order):

* Listing 1's triangular / diagonal solves from the converted band;
* the transposed solve with the band LU factors;
* the rectangular m x n band LU;
* band Cholesky, its solve and the band symmetry test;
* the fused detect-and-convert pass.

Shapes span the kernels' internal limits: ring register groups (K > 63), the
any-band kernel (K > 1023), the L^T pass's window chunks (kl > 64), the
Cholesky LDS window (kd <= 140) and its global-memory form, ragged sizes,
batches, empty inputs and the degenerate cases (zero diagonal, not positive
definite, exceeded caps)."""
import numpy as np
import pytest

import oracle
from paper_2608_22099_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_22099_amd import bandlu  # noqa: E402

DEV = "cuda:0"


def bits(x):
    return np.ascontiguousarray(x).view(np.uint64)


def same(a, b):
    """Bitwise equal, except that any NaN matches any NaN (the host and the
    device produce different NaN payloads for invalid operations)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.shape != b.shape:
        return False
    nan = np.isnan(a) & np.isnan(b)
    return bool(np.all((bits(a) == bits(b)) | nan))


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def band_T(n, kl, ku, seed, shift=0.0):
    return inputs.banded_dense(n, kl, ku, seed, shift=shift, check=False)


# ----------------------------------------------------------- triangular --
TRSV_SHAPES = [(1, 0, 0), (7, 0, 0), (300, 5, 0), (300, 0, 5), (1000, 63, 0), (1000, 0, 64),
               (777, 130, 0), (777, 0, 200), (1500, 1030, 0), (1500, 0, 1100), (64, 63, 0),
               (2, 1, 0), (2, 0, 1)]


@pytest.mark.parametrize("n,kl,ku", TRSV_SHAPES)
def test_trsv_bitwise(n, kl, ku):
    print(f"trsv n={n} kl={kl} ku={ku}", flush=True)
    T = band_T(n, kl, ku, 1100 + n + kl + 3 * ku, shift=2.0 * (kl + ku + 1))
    AB, _ = oracle.dense_to_band(T, kl, ku)
    B = np.random.default_rng(n + kl).standard_normal((3, n))
    ref = B.copy()
    info_o = oracle.band_trsv(AB, kl, ku, ref)
    ABg, Bg = gpu(AB), gpu(B)
    info = bandlu.band_trsv(ABg, kl, ku, Bg)
    torch.cuda.synchronize()
    assert int(info.cpu()[0]) == info_o
    assert same(Bg.cpu().numpy(), ref)


def test_trsv_zero_diagonal_and_batched():
    n, kl = 400, 9
    Ts = [band_T(n, kl, 0, 1200 + b, shift=20.0) for b in range(5)]
    Ts[2][123, 123] = 0.0
    Ts[4][0, 0] = 0.0
    ABs = np.stack([oracle.dense_to_band(T, kl, 0)[0] for T in Ts])
    B = np.random.default_rng(1201).standard_normal((5, 2, n))
    ref = B.copy()
    infos = [oracle.band_trsv(ABs[b], kl, 0, ref[b]) for b in range(5)]
    Bg = gpu(B)
    info = bandlu.band_trsv_batched(gpu(ABs), kl, 0, Bg)
    torch.cuda.synchronize()
    assert list(info.cpu().numpy()) == infos == [0, 0, 124, 0, 1]
    assert same(Bg.cpu().numpy(), ref)  # infinities and NaN included


# ------------------------------------------------------------ transposed --
GETRS_T_SHAPES = [(1, 0, 0), (2, 1, 0), (300, 3, 3), (500, 0, 7), (500, 7, 0), (1000, 16, 16),
                  (600, 70, 20), (800, 130, 100), (1200, 200, 900), (2000, 64, 64), (65, 64, 0)]


@pytest.mark.parametrize("n,kl,ku", GETRS_T_SHAPES)
def test_getrs_t_bitwise(n, kl, ku):
    print(f"getrs_t n={n} kl={kl} ku={ku}", flush=True)
    T = band_T(n, kl, ku, 1300 + n + kl + ku)
    AB, _ = oracle.dense_to_band(T, kl, ku)
    ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
    B = np.random.default_rng(1301 + n).standard_normal((2, n))
    ref = B.copy()
    oracle.gbtrs_t(AB, kl, ku, ipiv, ref)
    Bg = gpu(B)
    bandlu.band_getrs_t(gpu(AB), kl, ku, gpu(ipiv), Bg)
    torch.cuda.synchronize()
    assert same(Bg.cpu().numpy(), ref)


def test_getrs_t_batched_with_gpu_factors():
    """The transposed solve after the GPU factorisation, batched."""
    batch, n, kl, ku = 6, 300, 4, 6
    T = np.stack([band_T(n, kl, ku, 1400 + b) for b in range(batch)])
    ABg = bandlu.dense_to_band_batched(gpu(T), kl, ku)
    ipiv, info = bandlu.band_getrf_batched(ABg, kl, ku)
    B = np.random.default_rng(1401).standard_normal((batch, 3, n))
    Bg = gpu(B)
    bandlu.band_getrs_t_batched(ABg, kl, ku, ipiv, Bg)
    torch.cuda.synchronize()
    ABf, ipf, got = ABg.cpu().numpy(), ipiv.cpu().numpy(), Bg.cpu().numpy()
    for b in range(batch):
        ref = B[b].copy()
        oracle.gbtrs_t(ABf[b], kl, ku, ipf[b], ref)
        assert same(got[b], ref), b
        # and it solves A^T x = b
        r = T[b][:, :n] @ got[b].T - B[b].T
        assert np.abs(r).max() < 1e-9 * (1 + np.abs(got[b]).max())


# ----------------------------------------------------------- rectangular --
MN_SHAPES = [(1, 1, 0, 0), (3, 2, 2, 1), (2, 5, 1, 3), (300, 200, 10, 7), (200, 300, 6, 40),
             (500, 500, 20, 20), (130, 700, 129, 3), (700, 130, 300, 100)]


@pytest.mark.parametrize("m,n,kl,ku", MN_SHAPES)
def test_getrf_mn_bitwise(m, n, kl, ku):
    print(f"getrf_mn m={m} n={n} kl={kl} ku={ku}", flush=True)
    rng = np.random.default_rng(1500 + m + n)
    T = np.zeros((n, m))
    for j in range(n):
        lo, hi = max(0, j - ku), min(m - 1, j + kl)
        if lo <= hi:
            T[j, lo:hi + 1] = rng.standard_normal(hi - lo + 1)
    if min(m, n) > 4:
        T[min(m, n) // 2, :] = 0.0  # a zero column: info
    AB = oracle.dense_to_band_mn(T, m, kl, ku)
    ABg = gpu(AB)
    ipo, info_o, _ = oracle.gbtrf_mn(AB, m, kl, ku)
    ipiv, info = bandlu.band_getrf_mn(ABg, m, kl, ku)
    torch.cuda.synchronize()
    assert np.array_equal(ipiv.cpu().numpy(), ipo) and int(info.cpu()[0]) == info_o
    assert same(ABg.cpu().numpy(), AB)


def test_getrf_mn_batched():
    batch, m, n, kl, ku = 5, 150, 90, 8, 5
    ABs = []
    for b in range(batch):
        rng = np.random.default_rng(1600 + b)
        T = np.zeros((n, m))
        for j in range(n):
            lo, hi = max(0, j - ku), min(m - 1, j + kl)
            T[j, lo:hi + 1] = rng.standard_normal(hi - lo + 1)
        ABs.append(oracle.dense_to_band_mn(T, m, kl, ku))
    ABs = np.stack(ABs)
    ABg = gpu(ABs)
    ipiv, info = bandlu.band_getrf_mn_batched(ABg, m, kl, ku)
    torch.cuda.synchronize()
    for b in range(batch):
        ipo, info_o, _ = oracle.gbtrf_mn(ABs[b], m, kl, ku)
        assert np.array_equal(ipiv.cpu().numpy()[b], ipo) and int(info.cpu()[b]) == info_o
        assert same(ABg.cpu().numpy()[b], ABs[b])


# -------------------------------------------------------------- Cholesky --
def spd_T(n, kd, seed):
    rng = np.random.default_rng(seed)
    A = np.zeros((n, n))
    for d in range(1, kd + 1):
        v = rng.standard_normal(n - d)
        A[np.arange(d, n), np.arange(n - d)] = v
        A[np.arange(n - d), np.arange(d, n)] = v
    A[np.arange(n), np.arange(n)] = np.abs(A).sum(0) + 1.0
    return A  # symmetric: T = A


@pytest.mark.parametrize("n,kd", [(1, 0), (5, 0), (300, 1), (500, 8), (400, 63), (600, 140),
                                  (500, 141), (700, 200), (150, 149)])
def test_pbtrf_pbtrs_bitwise(n, kd):
    print(f"pbtrf n={n} kd={kd}", flush=True)
    A = spd_T(n, kd, 1700 + n + kd)
    AB = oracle.lower_band(A, kd)
    ABg = gpu(AB)
    info_o = oracle.pbtrf(AB, kd)
    info = bandlu.band_pbtrf(ABg, kd)
    torch.cuda.synchronize()
    assert int(info.cpu()[0]) == info_o == 0
    assert same(ABg.cpu().numpy(), AB)
    B = np.random.default_rng(1701).standard_normal((2, n))
    ref = B.copy()
    oracle.pbtrs(AB, kd, ref)
    Bg = gpu(B)
    bandlu.band_pbtrs(ABg, kd, Bg)
    torch.cuda.synchronize()
    assert same(Bg.cpu().numpy(), ref)


@pytest.mark.parametrize("kd", [3, 150])
def test_pbtrf_not_positive_definite(kd):
    n = 400
    A = spd_T(n, kd, 1800 + kd)
    A[250, 250] = -5.0
    AB = oracle.lower_band(A, kd)
    ABg = gpu(AB)
    info_o = oracle.pbtrf(AB, kd)
    info = bandlu.band_pbtrf(ABg, kd)
    torch.cuda.synchronize()
    assert int(info.cpu()[0]) == info_o > 0
    assert same(ABg.cpu().numpy(), AB)


def test_pbtrf_batched_and_ldab_from_conversion():
    """The lower layout read kd rows into dense_to_band(A, kd, 0)'s array."""
    batch, n, kd = 4, 256, 5
    As = [spd_T(n, kd, 1900 + b) for b in range(batch)]
    As[1][100, 100] = 0.0
    ABc = bandlu.dense_to_band_batched(gpu(np.stack(As)), kd, 0)  # ldab = 2kd+1
    low = ABc[:, :, kd:]  # lower layout, leading dimension 2kd+1
    info = bandlu.band_pbtrf_batched(low, kd)
    torch.cuda.synchronize()
    got = low.cpu().numpy()
    for b in range(batch):
        ref = oracle.lower_band(As[b], kd)
        io = oracle.pbtrf(ref, kd)
        assert int(info.cpu()[b]) == io
        assert same(got[b], ref)


def test_is_symmetric():
    A = spd_T(700, 6, 2000)
    assert int(bandlu.band_is_symmetric(gpu(A.T), 6).cpu()[0]) == oracle.is_symmetric_band(A.T.copy(), 6) == 1
    A2 = A.copy()
    A2[400, 403] = np.nextafter(A2[400, 403], 9.0)
    T2 = np.ascontiguousarray(A2.T)
    assert int(bandlu.band_is_symmetric(gpu(T2), 6).cpu()[0]) == oracle.is_symmetric_band(T2, 6) == 0
    A3 = A.copy()
    A3[10, 12], A3[12, 10] = 0.0, -0.0
    T3 = np.ascontiguousarray(A3.T)
    assert int(bandlu.band_is_symmetric(gpu(T3), 6).cpu()[0]) == 1


# --------------------------------------------------- fused detect+convert --
@pytest.mark.parametrize("n,kl,ku,klc,kuc,lda_pad", [
    (2048, 16, 16, 20, 30, 0),     # single-matrix flat kernel
    (4096, 3, 60, 3, 60, 0),       # caps equal to the bandwidths
    (1001, 5, 2, 9, 9, 0),         # odd n: column kernel
    (600, 40, 7, 64, 64, 3),       # padded lda: column kernel, scalar loads
    (2048, 0, 0, 4, 4, 0),         # diagonal
    (3000, 10, 300, 12, 299, 0),   # exceeds ku_cap
])
def test_detect_convert_bitwise(n, kl, ku, klc, kuc, lda_pad):
    print(f"detect_convert n={n} kl={kl} ku={ku} caps=({klc},{kuc})", flush=True)
    T = band_T(n, kl, ku, 2100 + n + kl + ku)
    # -0.0 between the band and the caps: must become +0.0 in the fill rows
    if ku + 1 < n:
        T[ku + 1, 0] = -0.0
    if lda_pad:
        T = np.concatenate([T, np.full((n, lda_pad), 7.0)], axis=1)
    kl_o, ku_o, ex_o, AB_o = oracle.detect_convert(T, klc, kuc)
    out, AB = bandlu.band_detect_convert(gpu(T)[:, :n] if not lda_pad else gpu(T), klc, kuc)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert o[2] == ex_o
    if ex_o:
        assert o[0] > klc or o[1] > kuc
        return
    assert (o[0], o[1]) == (kl_o, ku_o)
    view = bandlu.band_view(AB, klc, kuc, kl_o, ku_o).cpu().numpy()
    assert same(view, AB_o)


def test_detect_convert_batched_flat_and_lu():
    """Batch of n = 256 (flat batched kernel): the view of the batch maximum
    is dense_to_band_batched's output, and the band LU runs on it in place."""
    batch, n = 64, 256
    bands = [(4, 4), (2, 5), (4, 1), (3, 3)]
    T = np.stack([band_T(n, *bands[b % 4], 2200 + b) for b in range(batch)])
    out, dmax, AB = bandlu.band_detect_convert_batched(gpu(T), 8, 8)
    torch.cuda.synchronize()
    d = dmax.cpu().numpy()
    assert tuple(d) == (4, 5, 0)
    for b in range(batch):
        assert tuple(out.cpu().numpy()[b][:2]) == bands[b % 4]
    view = bandlu.band_view(AB, 8, 8, 4, 5)
    ref = np.stack([oracle.dense_to_band(T[b], 4, 5)[0] for b in range(batch)])
    assert same(view.cpu().numpy(), ref)
    ipiv, info = bandlu.band_getrf_batched(view, 4, 5)
    torch.cuda.synchronize()
    for b in (0, 17, 63):
        r = ref[b].copy()
        ipo, io, _ = oracle.gbtrf(r, 4, 5)
        assert np.array_equal(ipiv.cpu().numpy()[b], ipo)
        assert same(view.cpu().numpy()[b], r)


def test_detect_batched_batch_of_one_fills_dmax():
    T = band_T(2048, 7, 3, 2300)
    out, dmax = bandlu.band_detect_batched(gpu(T[None]))
    torch.cuda.synchronize()
    assert tuple(dmax.cpu().numpy()) == tuple(out.cpu().numpy()[0]) == (7, 3, 0)
