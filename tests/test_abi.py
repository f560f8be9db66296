"""The C ABI: the library loads, exports every symbol include/bandlu.h declares,
and validates arguments on the host (no GPU needed: validation returns before
any HIP call)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bandlu.h")
# (BANDLU_TEST_LIB: another build of the same library, e.g. one built with
# the host code under a sanitizer)
LIB = os.environ.get("BANDLU_TEST_LIB") or os.path.join(ROOT, "paper_2608_22099_amd", "libbandlu.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2608_22099_amd import build
        build.build()
    L = ctypes.CDLL(LIB)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    L.band_detect.argtypes = [vp, i64, i64, i64, i64, vp, vp]
    L.dense_to_band.argtypes = [vp, i64, i64, i64, i64, vp, i64, vp]
    L.band_getrf.argtypes = [i64, i64, i64, vp, i64, vp, vp, vp]
    L.band_getrf_batched.argtypes = [i64, i64, i64, vp, i64, i64, vp, i64, vp, i64, vp]
    L.band_getrf_batched_noalloc.argtypes = [i64, i64, i64, vp, i64, i64, vp, i64, vp, i64, vp]
    L.band_getrs.argtypes = [i64, i64, i64, i64, vp, i64, vp, vp, i64, vp]
    L.band_getrf_variant.argtypes = [i64, i64, i64, i64]
    L.band_getrf_ex.argtypes = [i64, i64, i64, vp, i64, i64, vp, i64, vp, i64, ctypes.c_int, vp]
    L.band_status_string.restype = ctypes.c_char_p
    L.band_last_error.restype = ctypes.c_char_p
    return L


def test_header_declares_the_path():
    names = declared_functions()
    for f in ["band_detect", "band_detect_batched", "dense_to_band", "dense_to_band_batched",
              "band_getrf", "band_getrf_batched", "band_getrs", "band_getrs_batched",
              "band_status_string", "band_last_error", "band_getrf_variant", "band_getrf_ex",
              "band_getrf_batched_noalloc"]:
        assert f in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for f in declared_functions():
        assert f in exported, f
        assert hasattr(lib, f)


def test_argument_validation(lib):
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert lib.band_detect(fake, -1, 1, -1, -1, fake, None) == -2
    assert lib.band_detect(fake, 10, 5, -1, -1, fake, None) == -3
    assert b"lda" in lib.band_last_error()
    assert lib.band_detect(fake, 10, 10, -1, -1, None, None) == -6
    assert lib.dense_to_band(fake, 10, 10, 10, 0, fake, 21, None) == -4
    assert lib.dense_to_band(fake, 10, 10, 2, 3, fake, 7, None) == -7
    assert lib.band_getrf(10, 2, 10, fake, 20, fake, fake, None) == -3
    assert lib.band_getrf(10, 2, 3, fake, 7, fake, fake, None) == -5
    assert lib.band_getrf(10, 2, 3, fake, 8, fake, None, None) == -7
    assert lib.band_getrf_batched(10, 2, 3, fake, 8, 79, fake, 10, fake, 2, None) == -6
    assert lib.band_getrf_batched(10, 2, 3, fake, 8, 80, fake, 9, fake, 2, None) == -8
    # the no-allocation form validates its arguments the same way
    nf = lib.band_getrf_batched_noalloc
    assert nf(10, 2, 3, fake, 8, 79, fake, 10, fake, 2, None) == -6
    assert nf(10, 2, 3, fake, 8, 80, fake, 9, fake, 2, None) == -8
    assert nf(10, 2, 3, fake, 7, 80, fake, 10, fake, 2, None) == -5
    assert nf(10, 2, 3, fake, 8, 80, fake, 10, None, 2, None) == -9
    assert b"noalloc" in lib.band_last_error()
    assert lib.band_getrs(10, 2, 3, -1, fake, 8, fake, fake, 10, None) == -4
    assert lib.band_getrs(10, 2, 3, 1, fake, 8, fake, fake, 9, None) == -9
    # the branches beyond the LU path validate on the host too
    L = lib
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    L.band_trsv.argtypes = [i64, i64, i64, i64, vp, i64, vp, i64, vp, vp]
    L.band_getrs_t.argtypes = [i64, i64, i64, i64, vp, i64, vp, vp, i64, vp]
    L.band_getrf_mn.argtypes = [i64, i64, i64, i64, vp, i64, vp, vp, vp]
    L.band_pbtrf.argtypes = [i64, i64, vp, i64, vp, vp]
    L.band_pbtrs.argtypes = [i64, i64, i64, vp, i64, vp, i64, vp]
    L.band_is_symmetric.argtypes = [vp, i64, i64, i64, vp, vp]
    L.band_detect_convert.argtypes = [vp, i64, i64, i64, i64, vp, vp, i64, vp]
    assert L.band_trsv(10, 2, 3, 1, fake, 8, fake, 10, fake, None) == -3  # not triangular
    assert L.band_trsv(10, 2, 0, 1, fake, 4, fake, 10, fake, None) == -6
    assert L.band_trsv(10, 0, 2, 1, fake, 3, fake, 9, fake, None) == -8
    assert L.band_getrs_t(10, 2, 3, 1, fake, 7, fake, fake, 10, None) == -6
    assert L.band_getrf_mn(5, 10, 5, 2, fake, 20, fake, fake, None) == -3  # kl > m-1
    assert L.band_getrf_mn(5, 10, 2, 10, fake, 20, fake, fake, None) == -4
    assert L.band_getrf_mn(5, 10, 2, 3, fake, 7, fake, fake, None) == -6
    assert L.band_pbtrf(10, 3, fake, 3, fake, None) == -4
    assert L.band_pbtrf(10, 10, fake, 11, fake, None) == -2
    assert L.band_pbtrs(10, 3, 1, fake, 4, fake, 9, None) == -7
    assert L.band_is_symmetric(fake, 10, 9, 2, fake, None) == -3
    assert L.band_detect_convert(fake, 10, 10, -1, 2, fake, fake, 10, None) == -4
    assert L.band_detect_convert(fake, 10, 10, 2, 2, fake, fake, 6, None) == -8
    # band_getrf_ex: argument 11 is the variant; a variant that cannot take the
    # sizes is refused before anything is enqueued
    assert lib.band_getrf_ex(10, 2, 3, fake, 8, 80, fake, 10, fake, 1, 9, None) == -11
    assert lib.band_getrf_ex(10, 0, 3, fake, 4, 40, fake, 10, fake, 1, 6, None) == -1001
    assert lib.band_getrf_ex(10, 0, 3, fake, 4, 40, fake, 10, fake, 1, 7, None) == -1001
    assert lib.band_getrf_ex(100, 2, 30, fake, 35, 3500, fake, 100, fake, 1, 7, None) == -1001
    assert lib.band_getrf_ex(100, 20, 22, fake, 63, 6300, fake, 100, fake, 1, 7, None) == -1001
    assert lib.band_getrf_ex(100, 3, 3, fake, 70, 7000, fake, 100, fake, 1, 7, None) == -1001
    assert lib.band_getrf_ex(10, 2, 3, fake, 8, 80, fake, 10, fake, 1, -1, None) == -11
    assert lib.band_getrf_ex(100, 40, 3, fake, 84, 8400, fake, 100, fake, 1, 1, None) == -1001
    assert b"variant 1" in lib.band_last_error()
    assert lib.band_getrf_ex(600, 300, 3, fake, 604, 0, fake, 600, fake, 1, 5, None) == -1001
    assert lib.band_getrf_ex(600, 300, 3, fake, 604, 0, fake, 600, fake, 1, 4, None) == -1001
    assert lib.band_status_string(-3) == b"invalid argument"
    assert lib.band_status_string(-1000).startswith(b"HIP")


def test_variant_selection(lib):
    W, G16, GEN, BLK, MF, SP, DG, WD = 1, 2, 3, 4, 5, 6, 7, 8
    assert lib.band_getrf_variant(1000, 3, 3, 1) == G16
    assert lib.band_getrf_variant(8192, 16, 16, 1) == DG
    assert lib.band_getrf_variant(300, 23, 17, 1) == DG
    assert lib.band_getrf_variant(300, 20, 22, 1) == SP
    assert lib.band_getrf_variant(300, 3, 24, 1) == DG
    assert lib.band_getrf_variant(300, 15, 24, 1) == SP
    assert lib.band_getrf_variant(300, 1, 24, 1) == DG
    # kl <= 6 beyond the diagonal-pivot kernel's reach: the lean window
    assert lib.band_getrf_variant(300, 2, 25, 1) == W
    assert lib.band_getrf_variant(300, 6, 40, 1) == W
    assert lib.band_getrf_variant(300, 6, 115, 1) == W
    assert lib.band_getrf_variant(300, 6, 116, 1) == BLK
    assert lib.band_getrf_variant(300, 7, 40, 1) == SP
    assert lib.band_getrf_variant(256, 4, 4, 63) == G16
    assert lib.band_getrf_variant(256, 5, 4, 63) == DG
    assert lib.band_getrf_variant(16384, 2, 64, 1) == W
    assert lib.band_getrf_variant(300, 15, 97, 1) == SP
    assert lib.band_getrf_variant(300, 0, 5, 1) == W
    assert lib.band_getrf_variant(300, 16, 97, 1) == BLK
    assert lib.band_getrf_variant(256, 4, 4, 4096) == G16
    # kl >= 32: the persistent kernel when the batch fits one launch of
    # co-resident workgroups (256 CUs assumed without a device), else one
    # launch per panel
    assert lib.band_getrf_variant(300, 40, 3, 1) == WD
    assert lib.band_getrf_variant(32768, 256, 256, 1) == WD
    assert lib.band_getrf_variant(300, 40, 3, 200) == MF
    assert lib.band_getrf_variant(300, 31, 90, 1) == BLK
    assert lib.band_getrf_variant(300, 20, 100, 1) == BLK
    assert lib.band_getrf_variant(300, 32, 0, 1) == WD
    assert lib.band_getrf_variant(2000, 300, 10, 1) == GEN
    assert lib.band_getrf_variant(-1, 0, 0, 1) == -1
