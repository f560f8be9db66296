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
