"""Host policy of the structure-aware LU: the decision of Listing 2.

Listing 2 detects the structure, and when the matrix is banded converts it and
factors it with the banded LU; otherwise it factors it as a dense matrix.  The
paper gives no body for its banded-structure test.  Here "banded" means that the
speedup constraint of Sec. II-B holds:

    I + C + f < F

with the four cost functions of Sec. II-A: I identifies the structure, C
converts the format, f runs the specialised algorithm, F the generic one.  They
can be evaluated two ways:

* as operation counts (``op_counts``): I = n^2 entries inspected, C =
  (2kl+ku+1) n band slots written, f = 2 n kl (kl+ku+1) flops of the banded LU
  with pivot fill, F = 2n^3/3 flops of the dense LU;
* as times measured on the device (``CostModel``): the detection and
  conversion rates, the banded LU time per column for the bandwidth class, and
  the dense LU (rocSOLVER getrf through torch) fitted as a + b n^3.

Both are monotone in kl and ku, so the largest bandwidths for which the
constraint can still hold are caps for the detection scan: once a bandwidth
exceeds its cap the banded branch cannot pay, and the scan may stop early
(the slowdown case of Sec. II-B, where T = I + F and the constraint I <= F
keeps the overhead bounded).

This module is host logic only: every step on the device runs in the HIP
kernels of libbandlu.so (through ``bandlu``), and the dense branch is the
generic algorithm F, rocSOLVER getrf through torch.
"""
from __future__ import annotations

import bisect
import time
from dataclasses import dataclass, field

import torch

from . import bandlu


# ----------------------------------------------------------- cost model --
def op_counts(n, kl, ku):
    """Operation counts of Sec. II-A for one n x n matrix with bandwidths (kl, ku):
    I = n^2 reads, C = (2kl+ku+1) n band slots, f = 2 n kl (kl+ku+1) flops,
    F = 2 n^3 / 3 flops."""
    I = n * n
    C = (2 * kl + ku + 1) * n
    f = 2 * n * kl * (kl + ku + 1)
    F = 2.0 * n ** 3 / 3.0
    return I, C, f, F


@dataclass
class CostModel:
    """Times (seconds) of the four cost functions, from rates measured on the
    device by ``measure``.

    detect_bps / convert_bps: bytes per second of the detection scan and the
        conversion (8 n^2 and 8 (in-band + ldab n) bytes);
    call_s: fixed cost of one library call (launch and queue);
    lu_probe: {(kl, ku): seconds per column} of band_getrf on random bands
        with row interchanges, measured at n = lu_probe_n;
    dense_a, dense_b: rocSOLVER getrf time a + b n^3.
    """
    detect_bps: float
    convert_bps: float
    call_s: float
    lu_probe: dict = field(default_factory=dict)
    lu_probe_n: int = 0
    dense_a: float = 0.0
    dense_b: float = 0.0

    def lu_time(self, n, kl, ku):
        """Band LU time: seconds per column of the smallest probed band that
        covers (kl, ku), times n (f is linear in n at fixed bands)."""
        best = None
        for (pl, pu), s in self.lu_probe.items():
            if pl >= kl and pu >= ku and (best is None or s < best):
                best = s
        if best is None:  # wider than every probe: scale the widest by the flop count
            (pl, pu), s = max(self.lu_probe.items(), key=lambda kv: kv[0][0] * (kv[0][0] + kv[0][1]))
            best = s * max(1.0, (kl * (kl + ku + 1)) / max(1, pl * (pl + pu + 1)))
        return self.call_s + best * n

    def times(self, n, kl, ku):
        ldab = 2 * kl + ku + 1
        I = self.call_s + 8.0 * n * n / self.detect_bps
        C = self.call_s + 8.0 * (n * (kl + ku + 1) + ldab * n) / self.convert_bps
        f = self.lu_time(n, kl, ku)
        F = self.dense_a + self.dense_b * float(n) ** 3
        return I, C, f, F

    @classmethod
    def measure(cls, device="cuda:0", seed=0, lu_n=2048,
                lu_bands=((1, 1), (4, 4), (16, 16), (3, 60), (31, 31), (64, 64), (128, 128),
                          (256, 256), (512, 512)),
                dense_sizes=(1024, 2048, 4096, 8192)):
        """Time the library's kernels and rocSOLVER getrf on synthetic inputs
        (seeded; about a second of device time)."""
        g = torch.Generator(device=device)
        g.manual_seed(seed)
        stream = torch.cuda.current_stream()

        def timed(fn, reps=3):
            fn()
            stream.synchronize()
            ts = []
            for _ in range(reps):
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record()
                fn()
                b.record()
                b.synchronize()
                ts.append(a.elapsed_time(b) * 1e-3)
            return sorted(ts)[len(ts) // 2]

        # detection and conversion rates on a 4096^2 band of 64 + 64
        n = 4096
        A = torch.zeros((n, n), dtype=torch.float64, device=device)
        for d in range(-64, 65):
            A.diagonal(d).copy_(torch.randn(n - abs(d), generator=g, device=device,
                                            dtype=torch.float64))
        out = torch.empty(3, dtype=torch.int64, device=device)
        t_small = timed(lambda: bandlu.band_detect(A[:64, :64].contiguous(), out=out))
        t_det = timed(lambda: bandlu.band_detect(A, out=out))
        AB = torch.empty((n, 2 * 64 + 64 + 1), dtype=torch.float64, device=device)
        t_conv = timed(lambda: bandlu.dense_to_band(A, 64, 64, AB=AB))
        call_s = t_small
        detect_bps = 8.0 * n * n / max(t_det - call_s, 1e-7)
        convert_bps = 8.0 * (n * 129 + n * 193) / max(t_conv - call_s, 1e-7)
        del A, AB

        # band LU per column (N(0,1) bands: row interchanges at most steps)
        probe = {}
        ipiv = torch.empty(lu_n, dtype=torch.int32, device=device)
        info = torch.empty(1, dtype=torch.int32, device=device)
        for kl, ku in lu_bands:
            kl, ku = min(kl, lu_n - 1), min(ku, lu_n - 1)
            ldab = 2 * kl + ku + 1
            src = torch.zeros((lu_n, ldab), dtype=torch.float64, device=device)
            src[:, kl:] = torch.randn((lu_n, kl + ku + 1), generator=g, device=device,
                                      dtype=torch.float64)
            work = torch.empty_like(src)

            def run():
                work.copy_(src)
                bandlu.band_getrf(work, kl, ku, ipiv=ipiv, info=info)

            t_copy = timed(lambda: work.copy_(src))
            probe[(kl, ku)] = max(timed(run) - t_copy - call_s, 0.0) / lu_n
            del src, work

        # dense LU: a + b n^3 by least squares
        xs, ys = [], []
        for m in dense_sizes:
            M = torch.randn((m, m), generator=g, device=device, dtype=torch.float64)
            ys.append(timed(lambda: torch.linalg.lu_factor(M), reps=2))
            xs.append(float(m) ** 3)
            del M
        k = len(xs)
        mx, my = sum(xs) / k, sum(ys) / k
        sxx = sum((x - mx) ** 2 for x in xs)
        b = sum((x - mx) * (y - my) for x, y in zip(xs, ys)) / sxx if sxx else ys[-1] / xs[-1]
        b = max(b, 1e-18)
        a = max(0.0, my - b * mx)
        return cls(detect_bps, convert_bps, call_s, probe, lu_n, a, b)

    def as_dict(self):
        return {"detect_GBs": self.detect_bps / 1e9, "convert_GBs": self.convert_bps / 1e9,
                "call_us": self.call_s * 1e6,
                "lu_ns_per_column": {f"{kl},{ku}": s * 1e9 for (kl, ku), s in self.lu_probe.items()},
                "lu_probe_n": self.lu_probe_n,
                "dense_lu_s": {"a": self.dense_a, "b_per_n3": self.dense_b}}


# ------------------------------------------------------------- predicates --
def speedup_predicate(n, kl, ku, model=None):
    """Sec. II-B speedup constraint I + C + f < F: take the banded branch.
    Operation counts without a model, measured times with one."""
    I, C, f, F = model.times(n, kl, ku) if model is not None else op_counts(n, kl, ku)
    return I + C + f < F


def slowdown_constraint(n, model=None):
    """Sec. II-B slowdown constraint I <= F: detection never costs more than
    the generic algorithm it may precede."""
    I, _, _, F = model.times(n, 0, 0) if model is not None else op_counts(n, 0, 0)
    return I <= F


def band_caps(n, model=None):
    """(kl_cap, ku_cap): the largest lower (upper) bandwidth for which the
    speedup constraint can still hold; -1 where every bandwidth can.  The
    costs only grow with kl and ku, so a matrix with kl > kl_cap or
    ku > ku_cap fails the constraint whatever its other bandwidth is."""
    def largest(ok):
        if n <= 1 or ok(n - 1):
            return -1
        if not ok(0):
            return 0
        lo, hi = 0, n - 1  # ok(lo), not ok(hi)
        while hi - lo > 1:
            mid = (lo + hi) // 2
            lo, hi = (mid, hi) if ok(mid) else (lo, mid)
        return lo
    kl_cap = largest(lambda b: speedup_predicate(n, b, 0, model))
    ku_cap = largest(lambda b: speedup_predicate(n, 0, b, model))
    return kl_cap, ku_cap


# ------------------------------------------------------- Listing 2 on GPU --
class BandLU:
    """Result of structure_aware_lu on the banded branch: the band factors,
    pivots and info of band_getrf, and the detected bandwidths."""

    branch = "banded"

    def __init__(self, AB, kl, ku, ipiv, info):
        self.AB, self.kl, self.ku, self.ipiv, self.info = AB, kl, ku, ipiv, info

    def solve(self, B):
        """Solve in place with band_getrs; B has shape (nrhs, ldb)."""
        return bandlu.band_getrs(self.AB, self.kl, self.ku, self.ipiv, B)


class DenseLU:
    """Result of structure_aware_lu on the dense branch: rocSOLVER getrf
    through torch (the generic algorithm F)."""

    branch = "dense"

    def __init__(self, LU, pivots, kl, ku, exceeded):
        self.LU, self.pivots = LU, pivots
        self.kl, self.ku, self.exceeded = kl, ku, exceeded

    def solve(self, B):
        """Solve in place; B has shape (nrhs, ldb) like BandLU.solve."""
        n = self.LU.shape[0]
        X = torch.linalg.lu_solve(self.LU, self.pivots, B[:, :n].transpose(0, 1))
        B[:, :n].copy_(X.transpose(0, 1))
        return B


def structure_aware_lu(A, model=None, caps=None, fused_caps=None):
    """Listing 2 on the GPU.

    A is an (n, lda) float64 device tensor holding the column-major matrix
    (``A[j, i]`` = element (i, j)).  Detection runs with early-exit caps from
    ``band_caps`` (or the given ``caps``); its (kl, ku, exceeded) come to the
    host in the path's one device-to-host copy.  If the speedup constraint
    holds the matrix is converted and factored with the banded LU (BandLU);
    otherwise it is factored densely with rocSOLVER (DenseLU).

    ``fused_caps`` = (kl_cap, ku_cap) takes the fused identify-and-convert
    pass instead: one read of the dense matrix packs the band of those caps
    while it detects (an (n, 2 kl_cap + ku_cap + 1) array), and the banded LU
    runs on the view of the detected band inside it.  If a cap is exceeded the
    path falls back to detection with the policy's caps.
    """
    n = A.shape[0]
    if fused_caps is not None:
        fkl, fku = (min(max(c, 0), max(n - 1, 0)) for c in fused_caps)
        out, ABc = bandlu.band_detect_convert(A, fkl, fku)
        kl, ku, exceeded = (int(v) for v in out.cpu())  # the one device->host copy
        if not exceeded and speedup_predicate(n, kl, ku, model):
            AB = bandlu.band_view(ABc, fkl, fku, kl, ku)
            ipiv, info = bandlu.band_getrf(AB, kl, ku)
            return BandLU(AB, kl, ku, ipiv, info)
        del ABc
    kl_cap, ku_cap = band_caps(n, model) if caps is None else caps
    out = bandlu.band_detect(A, kl_cap, ku_cap)
    kl, ku, exceeded = (int(v) for v in out.cpu())  # the one device->host copy
    if not exceeded and speedup_predicate(n, kl, ku, model):
        AB = bandlu.dense_to_band(A, kl, ku)
        ipiv, info = bandlu.band_getrf(AB, kl, ku)
        return BandLU(AB, kl, ku, ipiv, info)
    LU, piv = torch.linalg.lu_factor(A[:, :n].transpose(0, 1))
    return DenseLU(LU, piv, kl, ku, exceeded)


# ------------------------------------------------------- Listing 1 on GPU --
def structure_aware_solve(A, B, model=None, caps=None, spd=True):
    """The backslash dispatch of Listing 1 (Sec. I-C) on the GPU: solve
    A X = B in place on B (shape (nrhs, ldb), ``B[k, i]`` = row i of column k).

    Detection (with the caps of ``band_caps``) decides the branch, as
    Listing 1's element inspection does:
      * ku = 0 and/or kl = 0: diagonal, lower or upper triangular -- the band
        is converted and solved by substitution (band_trsv), no factorisation;
      * kl = ku and the band symmetric (``spd``): band Cholesky, the
        Cholesky case the paper names beside LU (Sec. II-B); a matrix that
        turns out not to be positive definite falls back to the LU branch;
      * otherwise, when the speedup constraint holds: banded LU and solve
        (Listing 2's branch), else the dense LU (rocSOLVER through torch).
    Returns the name of the branch taken."""
    n = A.shape[0]
    kl_cap, ku_cap = band_caps(n, model) if caps is None else caps
    out = bandlu.band_detect(A, kl_cap, ku_cap)
    kl, ku, exceeded = (int(v) for v in out.cpu())  # the one device->host copy
    if not exceeded and (kl == 0 or ku == 0):
        AB = bandlu.dense_to_band(A, kl, ku)
        bandlu.band_trsv(AB, kl, ku, B)
        return "diagonal" if kl == ku else ("upper" if kl == 0 else "lower")
    if not exceeded and spd and kl == ku and speedup_predicate(n, kl, ku, model):
        if int(bandlu.band_is_symmetric(A, kl).cpu()[0]):
            ABc = bandlu.dense_to_band(A, kl, 0)
            low = ABc[:, kl:]  # LAPACK's lower layout inside the converted band
            info = int(bandlu.band_pbtrf(low, kl).cpu()[0])
            if info == 0:
                bandlu.band_pbtrs(low, kl, B)
                return "cholesky"
    f = structure_aware_lu(A, model=model, caps=(kl_cap, ku_cap))
    f.solve(B)
    return f.branch


def timed_slowdown(A, model=None, reps=3):
    """The slowdown experiment of Sec. II-B on one dense-stored matrix: the
    time of the generic algorithm alone (T_generic = F) and with detection in
    front of it (T_struct^false = I + F), and their ratio.  Detection runs
    with the caps of ``band_caps`` (early exit) and, for comparison, as a
    full scan."""
    n = A.shape[0]
    caps = band_caps(n, model)
    out = torch.empty(3, dtype=torch.int64, device=A.device)
    M = A[:, :n].transpose(0, 1)
    stream = torch.cuda.current_stream()

    def ev_time(fn):
        fn()
        stream.synchronize()
        ts = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return sorted(ts)[len(ts) // 2]

    t_detect_cap = ev_time(lambda: bandlu.band_detect(A, caps[0], caps[1], out=out))
    det = [int(v) for v in out.cpu()]
    t_detect_full = ev_time(lambda: bandlu.band_detect(A, out=out))
    t_dense = ev_time(lambda: torch.linalg.lu_factor(M))
    return {"n": n, "caps": list(caps), "detect_capped_ms": t_detect_cap,
            "detect_capped_result": det, "detect_full_ms": t_detect_full, "dense_lu_ms": t_dense,
            "slowdown": (t_detect_cap + t_dense) / t_dense,
            "slowdown_full_scan": (t_detect_full + t_dense) / t_dense}
