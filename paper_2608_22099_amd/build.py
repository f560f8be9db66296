"""Build libbandlu.so (gfx950 only) from csrc/*.hip with hipcc.

Usage: python -m paper_2608_22099_amd.build [-j N] [--incremental]

Every translation unit is compiled for gfx950 with IEEE-exact floating point
(no fast-math, no fp contraction: every fused multiply-add in the kernels is
written explicitly) and with packed-fp32 instructions disabled.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbandlu.so")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

CFLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++20", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]


# kernels allowed some scratch (bytes per lane), by kernel name
SCRATCH_ALLOWED = {"getrf_wide_kernel": 256}


def _short(mangled):
    """The kernel's plain name inside a mangled symbol."""
    for name in SCRATCH_ALLOWED:
        if mangled and name in mangled:
            return name
    return mangled


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _headers_mtime():
    hs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hpp")]
    hs += [os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h")]
    return max((os.path.getmtime(h) for h in hs), default=0.0)


def _compile(src, incremental=False, hdr_mtime=0.0):
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    if incremental and os.path.exists(obj):
        t = os.path.getmtime(obj)
        if t >= os.path.getmtime(src) and t >= hdr_mtime:
            return obj, ""
    cmd = [HIPCC, *CFLAGS, "-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    # Every kernel must run without scratch memory: a register array indexed
    # at run time or a spill would fall back to it, which is slow, and a large
    # per-lane scratch size makes the runtime reserve memory for every wave slot.
    # The persistent wide-band kernel is the one exception, with a bound: a
    # few registers of its column steps spill (its launch has at most one
    # workgroup per CU, so the reserve is small).
    fn, bad = None, []
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            fn = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > SCRATCH_ALLOWED.get(_short(fn), 0):
            bad.append((fn, int(m.group(1))))
    if bad:
        raise RuntimeError(f"{src}: kernels use scratch memory: {bad[:5]}")
    err = "\n".join(l for l in r.stderr.splitlines() if "remark:" not in l and "packed-fp32" not in l)
    return obj, err


def build(jobs: int | None = None, verbose: bool = False, incremental: bool = False) -> str:
    """Compile every source (or, with incremental, only those whose object is
    older than the source or any header) and link the library."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4)))
    objs = []
    hdr = _headers_mtime()
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for obj, err in ex.map(lambda f: _compile(f, incremental, hdr), srcs):
            objs.append(obj)
            if verbose and err.strip():
                print(err, file=sys.stderr)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=None)
    ap.add_argument("-v", action="store_true")
    ap.add_argument("--incremental", action="store_true",
                    help="recompile only sources older than their object")
    a = ap.parse_args()
    print(build(a.j, a.v, a.incremental))
