"""Benchmark of the structure-aware banded LU path on one MI355X.

One step = the whole path of the paper's Listing 2 plus the solve, on one
matrix (or one batch) of synthetic dense-stored banded input already resident
in HBM: band_detect (with the early-exit caps of the speedup constraint) ->
one device-to-host copy of (kl, ku, exceeded) -> host policy (Sec. II-B
speedup constraint) -> dense_to_band -> band_getrf -> band_getrs.  A single
matrix that the persistent wide-band LU or the lean window LU (1 <= kl <= 6)
factors takes the two halves of band_gbsv for the last two (the same
results: "getrf" is the factorisation with the forward half of the solve
fused into that launch, "getrs" the backward half); other matrices and
batches call band_getrf(_batched) and band_getrs(_batched).

Prints ONE JSON line.  `value` is factorizations per second of the whole
path; per-call times come from HIP events on the stream every call is enqueued
on, and `roofline` rates the call that takes the most time.  Alongside:
detection with and without its early exit, the dense branch and the slowdown
experiment of Sec. II-B on dense inputs, the measured cost model against the
measured step, full-size parity of the timed factors against the CPU oracle,
and `cpu_baseline`, the oracle timed on a bounded sample of the workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
FP64_PEAK_TFLOPS = 78.6      # MI355X fp64, vector and matrix cores, TFLOP/s
DEFAULT_WORKLOAD = "n32768_kl256_ku256"
METRIC = "band-LU factorizations/s + detect GB/s (fraction of HBM/FP64 peak), 1 MI355X"
STEPS = ["detect", "convert", "getrf", "getrs"]


def kernel_costs(n, kl, ku, batch, fused=False):
    """Algorithmic bytes / flops per call of each step.  fused: the getrf step
    also runs the forward half of the solve (its multipliers, interchanges
    and right-hand side), and the getrs step is the backward half alone (U
    and the right-hand side)."""
    ldab = 2 * kl + ku + 1
    inband = sum(min(n - 1, j + kl) - max(0, j - ku) + 1 for j in range(n))
    costs = {
        "detect": {"bytes": 8.0 * n * n * batch},
        "convert": {"bytes": 8.0 * (inband + ldab * n) * batch},
        "getrf": {"bytes": (8.0 * (kl + ku + 1) * n + 8.0 * ldab * n + 4.0 * n) * batch,
                  "flops": 2.0 * n * kl * (kl + ku + 1) * batch},
        "getrs": {"bytes": (8.0 * ldab * n + 4.0 * n + 16.0 * n) * batch},
    }
    if fused:
        costs["getrf"]["bytes"] += (8.0 * kl * n + 4.0 * n + 16.0 * n) * batch
        costs["getrf"]["flops"] += 2.0 * n * kl * batch
        costs["getrs"]["bytes"] = (8.0 * (kl + ku + 1) * n + 16.0 * n) * batch
    return costs


# HIP sources each step's kernels are built from
STEP_SOURCES = {
    "detect": ["detect.hip", "common.hpp"],
    "convert": ["convert.hip", "common.hpp"],
    "getrf": ["getrf.hip", "getrf_win64.hpp", "getrf_win2.hpp", "getrf_lean64.hpp", "getrf_window.hpp",
              "getrf_g16.hpp",
              "getrf_split.hpp", "getrf_diag.hpp", "getrf_blocked.hip", "getrf_mfma.hip",
              "getrf_wide.hip", "chain.hip", "wave.hpp", "bufio.hpp", "common.hpp"],
    "getrs": ["getrs.hip", "getrs_ring.hpp", "getrs_ring.hip", "getrs_lane.hip", "chain.hip",
              "bufio.hpp", "common.hpp"],
}
# instantiation files of a step (one per parameter range), by name prefix
STEP_PREFIXES = {"getrf": ("getrf_win_g", "getrf_lean_fwd", "getrf_split_c", "getrf_diag_ku"),
                 "getrs": ("getrs_ring_fwd", "getrs_ring_bwd", "getrs_ring_div")}


def source_hash(step):
    """sha256 over the sources of one step: its counters are valid only for these."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_22099_amd", "csrc")
    files = [f for f in STEP_SOURCES[step] if os.path.exists(os.path.join(csrc, f))]
    for prefix in STEP_PREFIXES.get(step, ()):
        files += sorted(f for f in os.listdir(csrc) if f.startswith(prefix))
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per call of `kernel` on `workload` from the committed
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


def host_facts():
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    allowed = sorted(os.sched_getaffinity(0))
    return {"os_cpu_count": os.cpu_count(), "allowed_cores": len(allowed), "cpu_model": model}


def oracle_step(M, b):
    """One whole step of the oracle on one dense-stored matrix."""
    import oracle

    kl, ku, ex, _ = oracle.detect(M)
    AB, _ = oracle.dense_to_band(M, kl, ku)
    ipiv, info, _ = oracle.gbtrf(AB, kl, ku)
    x = oracle.gbtrs(AB, kl, ku, ipiv, b.copy())
    return kl, ku, AB, ipiv, info, x


def cpu_baseline(T, rhs, w, budget_s=12.0):
    """The oracle as it stands on whole steps of the workload, one thread
    pinned to one core.  Returns (entry, last oracle result) -- the latter
    feeds the full-size parity check of the timed GPU factors."""
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[0]
    batched = T.ndim == 3
    mats = T if batched else T[None]
    bs = rhs if batched else rhs[None]
    os.sched_setaffinity(0, {core})
    try:
        done, t0, last = 0, time.perf_counter(), None
        while True:
            last = oracle_step(mats[done % mats.shape[0]], bs[done % mats.shape[0]])
            done += 1
            el = time.perf_counter() - t0
            if el >= budget_s or (batched and done >= mats.shape[0]):
                break
    finally:
        os.sched_setaffinity(0, set(allowed))
    ent = {"value": done / el, "unit": "factorizations/s", "cores": 1, "kind": "oracle",
           "sample": f"{done} whole steps (detect+convert+gbtrf+gbtrs) of "
                     f"{'matrices of ' if batched else ''}the {w['name']} workload, one thread "
                     f"pinned to core {core}, {el:.1f} s",
           "host": host_facts()}
    return ent, (None if batched else last)


def cpu_batch_parallel(T, rhs):
    """The oracle on the whole batch spread over the allowed cores (its C code
    runs outside the interpreter lock, so threads run in parallel)."""
    workers = min(len(os.sched_getaffinity(0)), 16)
    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(lambda k: oracle_step(T[k], rhs[k]), range(T.shape[0])))
    el = time.perf_counter() - t0
    return {"value": T.shape[0] / el, "unit": "factorizations/s", "cores": workers,
            "sample": f"all {T.shape[0]} matrices, {workers} threads, {el:.1f} s"}


def full_size_parity(ABg, ipg, infg, xg, ref, kl, ku):
    """The timed GPU outputs against the oracle on the same input (its last
    cpu_baseline step): pivots and info exactly, factors bitwise or within
    the elementwise tolerance 1e-10 (entries that pass only against 1e-10
    times the largest entry of their column part are counted)."""
    _, _, ABo, ipo, info_o, xo = ref
    kv = kl + ku
    n, ldab = ABo.shape
    j = np.arange(n)[:, None]
    r = np.arange(ldab)[None, :]
    i = r - kv + j
    inside = (i >= 0) & (i < n) & (r <= kv + kl)
    U = inside & (r <= kv)
    L = inside & (r > kv)
    diff = np.abs(ABg - ABo)
    rel_ok = diff <= 1e-10 * np.abs(ABo)
    col = 0
    worst = 0.0
    for part in (U, L):
        scale = np.where(part, np.abs(ABo), 0.0).max(axis=1, keepdims=True)
        col += int(np.count_nonzero(part & ~rel_ok & (diff <= 1e-10 * scale)))
        with np.errstate(divide="ignore", invalid="ignore"):
            rel = np.where(part & (ABo != 0.0), diff / np.abs(ABo), 0.0)
        worst = max(worst, float(rel.max()))
    bitwise = bool(np.array_equal(ABg[inside].view(np.uint64), ABo[inside].view(np.uint64)))
    return {"ipiv_equal": bool(np.array_equal(ipg, ipo)), "info_equal": int(infg) == info_o,
            "factors_bitwise": bitwise, "factor_entries": int(np.count_nonzero(inside)),
            "max_rel_err": worst,
            "entries_within_tol_relative": int(np.count_nonzero(inside & rel_ok)),
            "entries_within_tol_column_scale_only": col,
            "entries_beyond_tol": int(np.count_nonzero(inside & ~rel_ok)) - col,
            "solution_max_rel_diff": float(np.abs(xg - xo).max() / np.abs(xo).max())}


def event_ms(torch, fn, reps=5):
    fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b))
    return float(np.median(ts))


def early_exit_timings(torch, bandlu, A, n, kl, ku, caps):
    """Detection at full size with and without its early exit: a full scan,
    caps at the detected bandwidths (no exit; the polling overhead), caps
    below them (exits), and a dense N(0,1) matrix of the same size with the
    policy's caps (the slowdown case)."""
    out = torch.empty(3, dtype=torch.int64, device=A.device)
    res = {}
    for name, (c0, c1) in [("full_scan", (-1, -1)), ("caps_at_bandwidths", (kl, ku)),
                           ("policy_caps", caps), ("caps_half", (kl // 2, ku // 2))]:
        t = event_ms(torch, lambda: bandlu.band_detect(A, c0, c1, out=out))
        res[name] = {"caps": [c0, c1], "ms": t, "result": [int(v) for v in out.cpu()],
                     "gbs_of_full_matrix": 8.0 * n * n / (t * 1e-3) / 1e9}
    res["overhead_caps_at_bandwidths"] = res["caps_at_bandwidths"]["ms"] / res["full_scan"]["ms"] - 1
    g = torch.Generator(device=A.device).manual_seed(123)
    D = torch.randn((n, n), generator=g, dtype=torch.float64, device=A.device)
    t = event_ms(torch, lambda: bandlu.band_detect(D, caps[0], caps[1], out=out))
    res["dense_input_policy_caps"] = {"caps": list(caps), "ms": t,
                                      "result": [int(v) for v in out.cpu()]}
    t = event_ms(torch, lambda: bandlu.band_detect(D, out=out))
    res["dense_input_full_scan"] = {"ms": t, "gbs": 8.0 * n * n / (t * 1e-3) / 1e9}
    del D
    return res


def extension_timings(torch, bandlu, A, n, kl, ku, ABf, ipf):
    """The branches beyond the LU path on the same workload, each on the GPU:
    the fused identify-and-convert pass against the two steps, the
    transposed solve and the upper triangular solve with the timed factors,
    a lower triangular band, band Cholesky and its solve on a symmetric
    positive definite band of the same n, and a rectangular band LU.  In-place
    calls get their inputs back before every rep, outside the timed region."""
    dev = A.device

    def timed(fn, restore=None, reps=5):
        ts = []
        for r in range(reps + 1):
            if restore is not None:
                restore()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            if r:
                ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    res = {}
    g = torch.Generator(device=dev).manual_seed(321)
    ldab = 2 * kl + ku + 1
    # fused identify-and-convert, caps at the bandwidths (the view is the array)
    out, out2 = (torch.empty(3, dtype=torch.int64, device=dev) for _ in range(2))
    ABc = torch.empty((n, ldab), dtype=torch.float64, device=dev)
    AB2 = torch.empty_like(ABc)
    t_f = timed(lambda: bandlu.band_detect_convert(A, kl, ku, AB=ABc, out=out))
    t_s = timed(lambda: (bandlu.band_detect(A, kl, ku, out=out2),
                         bandlu.dense_to_band(A, kl, ku, AB=AB2)))
    res["fused_detect_convert"] = {
        "caps": [kl, ku], "ms": t_f, "separate_detect_plus_convert_ms": t_s,
        "result": [int(v) for v in out.cpu()], "band_equal_to_separate": bool(torch.equal(ABc, AB2)),
        "algorithmic_gbs": (8.0 * n * n + 8.0 * ldab * n) / (t_f * 1e-3) / 1e9}
    del ABc, AB2
    b = torch.randn((1, n), generator=g, dtype=torch.float64, device=dev)
    x = torch.empty_like(b)
    # transposed solve and the upper triangular solve (U of the factors as a
    # band with kl = 0, ku = kl + ku) with the timed factors
    res["getrs_t_ms"] = timed(lambda: bandlu.band_getrs_t(ABf, kl, ku, ipf, x),
                              restore=lambda: x.copy_(b))
    res["trsv_upper_ms"] = timed(lambda: bandlu.band_trsv(ABf, 0, kl + ku, x),
                                 restore=lambda: x.copy_(b))
    ABl = torch.randn((n, 2 * kl + 1), generator=g, dtype=torch.float64, device=dev)
    ABl[:, kl] += 4.0 * (kl + 1)
    res["trsv_lower_ms"] = timed(lambda: bandlu.band_trsv(ABl, kl, 0, x), restore=lambda: x.copy_(b))
    del ABl
    # band Cholesky on an SPD band (strictly diagonally dominant, lower layout)
    for kd in (64, 140):
        L0 = torch.randn((n, kd + 1), generator=g, dtype=torch.float64, device=dev)
        L0[n - kd:, :] = 0.0
        for d in range(1, kd + 1):
            L0[n - d:, d] = 0.0
        row = L0[:, 1:].abs().sum(1)
        for d in range(1, kd + 1):
            row[d:] += L0[:n - d, d].abs()
        L0[:, 0] = row + 1.0
        L = L0.clone()
        info = torch.empty(1, dtype=torch.int32, device=dev)
        t_f = timed(lambda: bandlu.band_pbtrf(L, kd, info=info), restore=lambda: L.copy_(L0))
        t_s = timed(lambda: bandlu.band_pbtrs(L, kd, x), restore=lambda: x.copy_(b))
        res[f"pbtrf_kd{kd}"] = {"n": n, "kd": kd, "ms": t_f, "info": int(info.cpu()[0]),
                                "pbtrs_ms": t_s, "flops": float(n) * kd * (kd + 3)}
        del L0, L
    # rectangular band LU (one workgroup per matrix)
    m2, n2, k2 = 9216, 8192, 16
    R0 = torch.randn((n2, 3 * k2 + 1), generator=g, dtype=torch.float64, device=dev)
    Rm = R0.clone()
    res["getrf_mn"] = {"m": m2, "n": n2, "kl": k2, "ku": k2,
                       "ms": timed(lambda: bandlu.band_getrf_mn(Rm, m2, k2, k2),
                                   restore=lambda: Rm.copy_(R0))}
    return res


def slowdown_experiment(torch, policy, model, sizes=(8192, 16384, 32768)):
    """Sec. II-B slowdown on dense N(0,1) inputs: (I + F) / F with detection
    (early exit at the policy's caps, and as a full scan) in front of
    rocSOLVER getrf."""
    out = []
    for n in sizes:
        g = torch.Generator(device="cuda").manual_seed(1000 + n)
        D = torch.randn((n, n), generator=g, dtype=torch.float64, device="cuda")
        out.append(policy.timed_slowdown(D, model))
        del D
        torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense LU comparator")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip early-exit, slowdown and cost-model measurements")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 512 MiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only: every GPU box here has one "
                                   "GPU, and DESIGN.md describes how the path would shard",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2608_22099_amd import bandlu, inputs, policy

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
    caps = policy.band_caps(n) if batch == 1 else (-1, -1)
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

    # the kernels that run the forward solve inside the factorisation
    # (band_gbsv_lu): the persistent wide-band LU, and the lean window LU
    # (the window variant for 1 <= kl <= 6) with one right-hand side
    variant1 = bandlu.band_getrf_variant(n, kl, ku, 1)
    fused = batch == 1 and (variant1 == "wide" or (variant1 == "window" and 1 <= kl <= 6))

    def step(timed):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)] if timed else None
        if timed:
            ev[0].record()
        if batch == 1:
            bandlu.band_detect(A, caps[0], caps[1], out=det)
            src = det
        else:
            bandlu.band_detect_batched(A, out=det, dmax=dmax)
            src = dmax
        if timed:
            ev[1].record()
        kl_d, ku_d, ex = (int(v) for v in src.cpu())  # the one device->host crossing
        assert (kl_d, ku_d, ex) == (kl, ku, 0)
        assert policy.speedup_predicate(n, kl_d, ku_d)
        if timed:
            ev[2].record()
        if batch == 1:
            bandlu.dense_to_band(A, kl_d, ku_d, AB=AB)
        else:
            bandlu.dense_to_band_batched(A, kl_d, ku_d, AB=AB)
        x.copy_(b0)
        if timed:
            ev[3].record()
        # a matrix that the persistent wide-band LU or the lean window LU
        # factors: the factorisation with the forward half of the solve fused
        # into it, then the backward half (band_getrf + band_getrs, the same
        # results); otherwise the two calls themselves
        if fused:
            bandlu.band_gbsv_lu(AB, kl_d, ku_d, x, ipiv=ipiv, info=info)
        elif batch == 1:
            bandlu.band_getrf(AB, kl_d, ku_d, ipiv=ipiv, info=info)
        else:
            bandlu.band_getrf_batched(AB, kl_d, ku_d, ipiv=ipiv, info=info)
        if timed:
            ev[4].record()
        if fused:
            bandlu.band_gbsv_back(AB, kl_d, ku_d, x)
        elif batch == 1:
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
    acc = {k: 0.0 for k in STEPS}
    for ev in events:
        acc["detect"] += ev[0].elapsed_time(ev[1])
        acc["convert"] += ev[2].elapsed_time(ev[3])
        acc["getrf"] += ev[3].elapsed_time(ev[4])
        acc["getrs"] += ev[4].elapsed_time(ev[5])
    avg = {k: acc[k] / args.steps for k in STEPS}
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = batch * 1e3 / ms_per_step  # factorizations per second, whole path
    timed_out = (AB.cpu().numpy(), ipiv.cpu().numpy(), info.cpu().numpy(), x.cpu().numpy())

    costs = kernel_costs(n, kl, ku, batch, fused)
    kernels = {k: roofline_entry(k, avg[k], costs[k]) for k in STEPS}
    dom = max(STEPS, key=lambda k: avg[k])
    d = kernels[dom]
    variant = bandlu.band_getrf_variant(n, kl, ku, batch)
    if "flops" in costs[dom] and costs[dom]["flops"] / costs[dom]["bytes"] > \
            FP64_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma" if variant in ("wide", "blocked_mfma") else "alu",
                "achieved": d["tflops"], "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": d["frac_fp64"]}
    else:
        roof = {"bound": "hbm", "achieved": d["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": d["frac_hbm"]}
    roof["traffic"] = measured_traffic(dom, args.workload)
    roof["kernel"] = dom
    for k in STEPS:
        kernels[k]["traffic_bytes"] = measured_traffic(k, args.workload)
        kernels[k]["algorithmic_bytes"] = costs[k]["bytes"]
    kernels["getrf"]["variant"] = variant
    kernels["getrs"]["variant"] = bandlu.band_getrs_variant(n, kl, ku, 1, batch)
    if fused:
        kernels["getrf"]["entry"] = "band_gbsv_lu (factorisation + forward half of the solve)"
        kernels["getrs"]["entry"] = "band_gbsv_back (backward half of the solve)"

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
        "detect_caps": list(caps),
    }
    model = None
    if not args.no_extras:
        model = policy.CostModel.measure(str(dev))
        I, C, f, F = model.times(n, kl, ku)
        out["cost_model"] = model.as_dict()
        out["cost_model_vs_measured_ms"] = {
            "predicted": {"I": I * 1e3, "C": C * 1e3, "f": f * 1e3, "F": F * 1e3},
            "measured": {"I": avg["detect"], "C": avg["convert"], "f": avg["getrf"]},
            "speedup_constraint_model": bool(I + C + f < F),
            "speedup_constraint_op_counts": bool(policy.speedup_predicate(n, kl, ku))}
        if batch == 1:
            out["early_exit"] = early_exit_timings(torch, bandlu, A, n, kl, ku, caps)
            out["extensions"] = extension_timings(torch, bandlu, A, n, kl, ku, AB, ipiv)
    if not args.no_dense and batch == 1:
        M = A[:, :n].transpose(0, 1)
        t_dense = event_ms(torch, lambda: torch.linalg.lu_factor(M), reps=3)
        t_struct = avg["detect"] + avg["convert"] + avg["getrf"]
        out["dense_lu_ms"] = t_dense
        out["speedup_vs_dense_lu"] = t_dense / ms_per_step
        out["speedup_vs_dense_lu_kernels_only"] = t_dense / t_struct
        if not args.no_extras:
            del M
            torch.cuda.empty_cache()
            out["slowdown_dense_inputs"] = slowdown_experiment(torch, policy, model)
    del A
    torch.cuda.empty_cache()
    if not args.no_cpu:
        ent, ref = cpu_baseline(T if batch == 1 else T[:256], rhs if batch == 1 else rhs[:256], w)
        if batch > 1:
            ent["batch_parallel"] = cpu_batch_parallel(T, rhs)
        out["cpu_baseline"] = ent
        if ref is not None:
            ABg, ipg, infg, xg = timed_out
            out["parity_full_size"] = full_size_parity(ABg, ipg, infg[0], xg, ref, kl, ku)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
