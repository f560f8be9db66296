"""Benchmark of the structure-aware banded LU path on one MI355X.

One step = the whole path of the paper's Listing 2 plus the solve, on one
matrix (or one batch) of synthetic dense-stored banded input already resident
in HBM: band_detect -> one device-to-host copy of (kl, ku, exceeded) -> host
policy (speedup constraint) -> dense_to_band -> band_getrf -> band_getrs.

Prints ONE JSON line.  `value` is factorizations per second of the whole
path; per-kernel times come from HIP events on the stream the kernels run on,
and `roofline` rates the kernel that takes the most time.  `cpu_baseline`
times the CPU oracle on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
FP64_PEAK_TFLOPS = 78.6      # MI355X fp64 (vector and matrix), TFLOP/s
DEFAULT_WORKLOAD = "n8192_kl16_ku16"
METRIC = "band-LU factorizations/s + detect GB/s (fraction of HBM/FP64 peak), 1 MI355X"


def kernel_costs(n, kl, ku, batch):
    """Algorithmic bytes / flops per launch of each step."""
    ldab = 2 * kl + ku + 1
    inband = sum(min(n - 1, j + kl) - max(0, j - ku) + 1 for j in range(n)) if n < 70000 else n * (kl + ku + 1)
    return {
        "detect": {"bytes": 8.0 * n * n * batch},
        "convert": {"bytes": 8.0 * (inband + ldab * n) * batch},
        "getrf": {"bytes": (8.0 * (kl + ku + 1) * n + 8.0 * ldab * n + 4.0 * n) * batch,
                  "flops": 2.0 * n * kl * (kl + ku + 1) * batch},
        "getrs": {"bytes": (8.0 * ldab * n + 4.0 * n + 16.0 * n) * batch},
    }


# HIP sources each step's kernels are built from
STEP_SOURCES = {
    "detect": ["detect.hip", "common.hpp"],
    "convert": ["convert.hip", "common.hpp"],
    "getrf": ["getrf.hip", "getrf_win64.hpp", "getrf_win2.hpp", "getrf_window.hpp", "getrf_g16.hpp",
              "getrf_split.hpp", "getrf_diag.hpp", "getrf_blocked.hip", "getrf_mfma.hip", "wave.hpp",
              "bufio.hpp", "common.hpp"],
    "getrs": ["getrs.hip", "getrs_ring.hpp", "getrs_ring.hip", "getrs_lane.hip", "bufio.hpp",
              "common.hpp"],
}
# instantiation files of a step (one per parameter range), by name prefix
STEP_PREFIXES = {"getrf": ("getrf_win_g", "getrf_split_c", "getrf_diag_ku"),
                 "getrs": ("getrs_ring_fwd", "getrs_ring_bwd")}


def source_hash(step):
    """sha256 over the sources of one step: its counters are valid only for these."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_22099_amd", "csrc")
    files = list(STEP_SOURCES[step])
    for prefix in STEP_PREFIXES.get(step, ()):
        files += sorted(f for f in os.listdir(csrc) if f.startswith(prefix))
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the
    same counter on a plain copy of known size), or None when there is no
    summary or the kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"counters_{workload}.md")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ":" in line:
                k, v = line[2:].split(":", 1)
                vals[k.strip()] = v.strip().strip("`")
    if vals.get(f"{kernel}.source_sha256") != source_hash(kernel):
        return None
    try:
        fetch = float(vals[f"{kernel}.FETCH_SIZE_KiB"])
        write = float(vals[f"{kernel}.WRITE_SIZE_KiB"])
        copy_bytes = float(vals["copy.bytes"])
        fscale = copy_bytes / (float(vals["copy.FETCH_SIZE_KiB"]) * 1024.0)
        wscale = copy_bytes / (float(vals["copy.WRITE_SIZE_KiB"]) * 1024.0)
    except (KeyError, ValueError, ZeroDivisionError):
        return None
    return fetch * 1024.0 * fscale + write * 1024.0 * wscale


def copy_calibration():
    """A plain device copy of known size, profiled beside the path to scale
    FETCH_SIZE / WRITE_SIZE into bytes."""
    import torch

    n = 64 * 1024 * 1024  # 512 MiB of doubles
    a = torch.ones(n, dtype=torch.float64, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n * 8, "launches": 3}))


def roofline_entry(name, t_ms, cost):
    t = t_ms * 1e-3
    gbs = cost["bytes"] / t / 1e9
    ent = {"kernel": name, "avg_ms": t_ms, "gbs": gbs, "frac_hbm": gbs / HBM_PEAK_GBS}
    if "flops" in cost:
        tf = cost["flops"] / t / 1e12
        ent["tflops"] = tf
        ent["frac_fp64"] = tf / FP64_PEAK_TFLOPS
        ent["arith_intensity"] = cost["flops"] / cost["bytes"]
    return ent


def cpu_baseline(T, w, budget_s=12.0):
    """The oracle as it stands, one thread, on whole steps of the workload."""
    import oracle

    n, kl, ku = w["n"], w["kl"], w["ku"]
    mats = T if T.ndim == 3 else T[None]
    done, t0 = 0, time.perf_counter()
    b = np.random.default_rng(0).standard_normal((1, n))
    while True:
        M = mats[done % mats.shape[0]]
        kl_d, ku_d, ex, _ = oracle.detect(M)
        AB, _ = oracle.dense_to_band(M, kl_d, ku_d)
        ipiv, info, _ = oracle.gbtrf(AB, kl_d, ku_d)
        oracle.gbtrs(AB, kl_d, ku_d, ipiv, b.copy())
        done += 1
        el = time.perf_counter() - t0
        if el >= budget_s or (mats.shape[0] > 1 and done >= mats.shape[0]):
            break
    per_fact = el / done
    return {"value": 1.0 / per_fact, "unit": "factorizations/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} whole factorizations (detect+convert+gbtrf+gbtrs) of "
                      f"{'matrices of ' if T.ndim == 3 else ''}the {w['name']} workload, "
                      f"single thread, {el:.1f} s"}


def dense_comparator(A_dev, n, reps=3):
    """rocSOLVER getrf through torch on the same dense matrix (generic branch F)."""
    import torch

    M = A_dev[:, :n].transpose(0, 1)
    torch.linalg.lu_factor(M)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        torch.linalg.lu_factor(M)
        torch.cuda.synchronize()
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts)) * 1e3


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense LU comparator")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 512 MiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; the path is a single-GPU "
                                   "kernel pipeline (see DESIGN.md for how it would shard)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2608_22099_amd import bandlu, inputs

    w = dict(inputs.WORKLOADS[args.workload])
    w["name"] = args.workload
    n, kl, ku, batch = w["n"], w["kl"], w["ku"], w["batch"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if batch == 1:
        T = inputs.workload_matrix(args.workload)
        rhs = inputs.workload_rhs(args.workload)
    else:
        T = inputs.workload_batch(args.workload)
        rhs = np.stack([inputs.workload_rhs(args.workload, b) for b in range(batch)])
    A = torch.from_numpy(T).to(dev)
    b0 = torch.from_numpy(rhs).to(dev)
    x = torch.empty_like(b0)
    ldab = 2 * kl + ku + 1
    if batch == 1:
        AB = torch.empty((n, ldab), dtype=torch.float64, device=dev)
        ipiv = torch.empty(n, dtype=torch.int32, device=dev)
        info = torch.empty(1, dtype=torch.int32, device=dev)
        det = torch.empty(3, dtype=torch.int64, device=dev)
    else:
        AB = torch.empty((batch, n, ldab), dtype=torch.float64, device=dev)
        ipiv = torch.empty((batch, n), dtype=torch.int32, device=dev)
        info = torch.empty(batch, dtype=torch.int32, device=dev)
        det = torch.empty((batch, 3), dtype=torch.int64, device=dev)
        dmax = torch.empty(3, dtype=torch.int64, device=dev)

    names = ["detect", "convert", "getrf", "getrs"]
    acc = {k: 0.0 for k in names}

    def step(timed):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)] if timed else None
        if timed:
            ev[0].record()
        if batch == 1:
            bandlu.band_detect(A, out=det)
            src = det
        else:
            bandlu.band_detect_batched(A, out=det, dmax=dmax)
            src = dmax
        if timed:
            ev[1].record()
        kl_d, ku_d, ex = (int(v) for v in src.cpu())  # the one device->host crossing
        assert (kl_d, ku_d, ex) == (kl, ku, 0)
        assert bandlu.speedup_predicate(n, kl_d, ku_d)
        if timed:
            ev[2].record()
        if batch == 1:
            bandlu.dense_to_band(A, kl_d, ku_d, AB=AB)
        else:
            bandlu.dense_to_band_batched(A, kl_d, ku_d, AB=AB)
        if timed:
            ev[3].record()
        if batch == 1:
            bandlu.band_getrf(AB, kl_d, ku_d, ipiv=ipiv, info=info)
        else:
            bandlu.band_getrf_batched(AB, kl_d, ku_d, ipiv=ipiv, info=info)
        if timed:
            ev[4].record()
        x.copy_(b0)
        if batch == 1:
            bandlu.band_getrs(AB, kl_d, ku_d, ipiv, x)
        else:
            bandlu.band_getrs_batched(AB, kl_d, ku_d, ipiv, x)
        if timed:
            ev[5].record()
        return ev

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    events = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        events.append(step(True))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for ev in events:
        acc["detect"] += ev[0].elapsed_time(ev[1])
        acc["convert"] += ev[2].elapsed_time(ev[3])
        acc["getrf"] += ev[3].elapsed_time(ev[4])
        acc["getrs"] += ev[4].elapsed_time(ev[5])
    avg = {k: acc[k] / args.steps for k in names}
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = batch * 1e3 / ms_per_step  # factorizations per second, whole path

    costs = kernel_costs(n, kl, ku, batch)
    kernels = {k: roofline_entry(k, avg[k], costs[k]) for k in names}
    dom = max(names, key=lambda k: avg[k])
    d = kernels[dom]
    if "flops" in costs[dom] and costs[dom]["flops"] / costs[dom]["bytes"] > \
            FP64_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "alu", "achieved": d["tflops"], "peak": FP64_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": d["frac_fp64"], "traffic": None}
    else:
        roof = {"bound": "hbm", "achieved": d["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": d["frac_hbm"], "traffic": None}
    roof["kernel"] = dom
    tb = measured_traffic(dom, args.workload)
    roof["traffic"] = tb
    for k in names:
        t = measured_traffic(k, args.workload)
        kernels[k]["traffic_bytes"] = t
        kernels[k]["algorithmic_bytes"] = costs[k]["bytes"]

    out = {
        "metric": METRIC, "value": value, "unit": "factorizations/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded dense-stored banded fp64, see DESIGN.md input recipe)",
        "config": {"workload": args.workload, "n": n, "kl": kl, "ku": ku, "batch": batch,
                   "nrhs": 1, "parallelism": "single GPU"},
        "roofline": roof,
        "detect_gbs": kernels["detect"]["gbs"],
        "detect_frac_hbm": kernels["detect"]["frac_hbm"],
        "getrf_gflops_effective": costs["getrf"]["flops"] / (avg["getrf"] * 1e-3) / 1e9,
        "kernels": kernels,
    }
    if not args.no_dense and batch == 1:
        t_dense = dense_comparator(A, n)
        t_struct = avg["detect"] + avg["convert"] + avg["getrf"]
        out["dense_lu_ms"] = t_dense
        out["speedup_vs_dense_lu"] = t_dense / ms_per_step
        out["speedup_vs_dense_lu_kernels_only"] = t_dense / t_struct
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(T if batch == 1 else T[:256], w)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
