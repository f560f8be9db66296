"""Planted mistakes in the oracle (on the CPU): each mutant of the oracle's C
source must make the pin suite fail, which shows that the pins can tell a
plausible slip (dropped term, wrong sign, wrong index, transposed operand)
from the correct arithmetic."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "bandlu_oracle.c")

MUTANTS = {
    "update_sign": ("fma(-AT(j + t, j), u, AT(j + t, c))", "fma(AT(j + t, j), u, AT(j + t, c))"),
    "pivot_tie_break": ("if (fabs(AT(j + t, j)) > dmax)", "if (fabs(AT(j + t, j)) >= dmax)"),
    "fill_extent": ("ju = imax(ju, imin(j + ku + p, n - 1));", "ju = imax(ju, imin(j + ku, n - 1));"),
    "dropped_swap_half": ("AT(j + p, c) = tmp;", "(void)tmp;"),
    "detect_transposed": ("if (i - j > kl) kl = i - j;", "if (j - i > kl) kl = j - i;"),
    "convert_offset": ("int64_t i = r - kl - ku + j; /* matrix row of this slot */",
                       "int64_t i = r - kl - ku + j + 1;"),
    "solve_backward_range": ("for (int64_t i = imax(0, j - kv); i < j; ++i) b[i]",
                             "for (int64_t i = imax(0, j - kv + 1); i < j; ++i) b[i]"),
    "solve_forward_swap": ("b[l] = b[j];\n                    b[j] = tmp;", "(void)tmp;"),
    "scale_by_division": ("AT(j + t, j) = AT(j + t, j) * r;", "AT(j + t, j) = AT(j + t, j) / piv;"),
    "info_index": ("*info = (int32_t)(j + 1);\n        }\n    }\n#undef AT\n    if (flops)",
                   "*info = (int32_t)(j);\n        }\n    }\n#undef AT\n    if (flops)"),
    "tiny_pivot_reciprocal": ("for (int64_t t = 1; t <= km; ++t) AT(j + t, j) = AT(j + t, j) / piv;",
                              "for (int64_t t = 1; t <= km; ++t) AT(j + t, j) = AT(j + t, j) * (1.0 / piv);"),
    "gepp_tiny_pivot_reciprocal": ("for (int64_t i = k + 1; i < n; ++i) A[i + k * lda] /= piv;",
                                   "for (int64_t i = k + 1; i < n; ++i) A[i + k * lda] *= 1.0 / piv;"),
    "tiny_pivot_threshold": ("if (fabs(piv) >= DBL_MIN) {\n                    double r = 1.0 / piv;",
                             "if (fabs(piv) > 0.0) {\n                    double r = 1.0 / piv;"),
    "fill_zeroing": ("r < kl; ++r) AB[r + c * ldab] = 0.0;", "r < kl; ++r) (void)0;"),
    # triangular / diagonal solve
    "trsv_lower_range": ("for (int64_t i = j + 1; i <= imin(n - 1, j + kl); ++i)\n                    b[i]",
                         "for (int64_t i = j + 1; i <= imin(n - 1, j + kl - 1); ++i)\n                    b[i]"),
    "trsv_upper_no_divide": ("b[j] = b[j] / AT(j, j);\n                for (int64_t i = imax(0, j - ku); i < j; ++i)",
                             "b[j] = b[j];\n                for (int64_t i = imax(0, j - ku); i < j; ++i)"),
    "trsv_info_index": ("if (AT(j, j) == 0.0) {\n            *info = (int32_t)(j + 1);",
                        "if (AT(j, j) == 0.0) {\n            *info = (int32_t)(j);"),
    # transposed solve
    "gbtrs_t_transposed_operand": ("b[j] = fma(-AT(i, j), b[i], b[j]);", "b[j] = fma(-AT(j, i), b[i], b[j]);"),
    "gbtrs_t_lpass_index": ("b[j] = fma(-AT(j + t, j), b[j + t], b[j]);",
                            "b[j] = fma(-AT(j + t, j), b[j + t - 1], b[j]);"),
    "gbtrs_t_dropped_swap": ("b[l] = b[j];\n                    b[j] = bl;", "(void)bl;"),
    # rectangular LU
    "gbtrf_mn_candidates": ("const int64_t km = imin(kl, m - 1 - j);", "const int64_t km = imin(kl, n - 1 - j);"),
    "gbtrf_mn_extent": ("ju = imax(ju, imin(n - 1, j + ku + p));", "ju = imax(ju, imin(n - 1, j + ku));"),
    # band Cholesky
    "pbtrf_update_operand": ("LT(i, c) = fma(-LT(i, j), LT(c, j), LT(i, c));",
                             "LT(i, c) = fma(-LT(i, j), LT(i, j), LT(i, c));"),
    "pbtrf_no_sqrt": ("const double d = sqrt(d0);", "const double d = d0;"),
    "pbtrf_pd_test": ("if (!(d0 > 0.0)) {", "if (d0 < 0.0) {"),
    "pbtrs_backward_transpose": ("b[i] = fma(-LT(j, i), b[j], b[i]);", "b[i] = fma(-LT(i, j), b[j], b[i]);"),
    "symmetric_compare": ("if (!(A[i + j * lda] == A[j + i * lda])) return 0;",
                          "if (!(A[i + j * lda] == A[i + j * lda])) return 0;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                           "-o", str(so), str(mpath), "-lm"])
    env = dict(os.environ, BANDLU_ORACLE_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
