#!/usr/bin/env python3
"""Throughput of costa_transform on one MI355X.

One step = one costa_transform (or costa_transform_batched) call: the direct
path, then pack and unpack-transform of every wave, over synthetic seeded
inputs already resident in HBM.  The plan (grid overlay, volume kernel,
relabeling, rectangles) is built before the timed region and cached.

Metric: effective GB/s = model bytes per step / time per step, with model
bytes = read B + read A (beta != 0) + write A + 2 x message bytes (each
message element is written by the pack and read by the unpack).

Also reported: the median and minimum step time (events between the timed
steps), and the bytes a transform without message staging would move
(read B + read A if beta != 0 + write A).

Prints one JSON line.  The default workload is the ScaLAPACK-style block-size
change: fp64 16384 x 16384, 4x4 process grid, 128x128 -> 256x256 blocks,
identity op, alpha = 1, beta = 0, relabeling on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
METRIC = "effective GB/s of costa_transform (and % of HBM peak) per config, 1 MI355X"
KINDS = ["pack", "unpack", "direct"]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    # the kernels and what decides their launches (rectangles, groups, order)
    for f in ("paper_2106_06601_amd/csrc/kernels.hip", "paper_2106_06601_amd/csrc/internal.hpp",
              "paper_2106_06601_amd/csrc/plan.cpp", "paper_2106_06601_amd/csrc/api.cpp"):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(workload: str, kernel: str, launches_per_step: float):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when it is missing or was taken from a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"counters_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    return d.get("hbm_bytes_per_launch")


def describe(w) -> dict:
    def lay(s):
        if s.kind == "block_cyclic":
            return (f"block-cyclic {s.prow}x{s.pcol} grid, {s.mb}x{s.nb} blocks, {s.rank_order}-major ranks, "
                    f"{s.block_order}-major storage")
        return (f"general grid {len(s.row_splits) - 1}x{len(s.col_splits) - 1} blocks over {s.nranks} ranks, "
                f"{s.block_order}-major storage")
    it = w.items[0]
    return {"workload": w.name, "description": w.description, "dtype": w.dtype, "pairs": len(w.items),
            "A": f"{it.A.nrows}x{it.A.ncols}", "source": lay(it.B), "target": lay(it.A),
            "ops": "".join(x.op for x in w.items), "alpha": str(it.alpha), "beta": str(it.beta),
            "relabel": w.relabel, "P": it.A.nranks}


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, sigma, model_bytes_per_elem: float, target_s: float, threads: int):
    """The CPU oracle on bands of target rows of pair 0, run by `threads`
    threads at once (the oracle's C loop runs outside the GIL)."""
    import threading
    import numpy as np
    import oracle
    import synth
    it = w.items[0]
    OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
    P = it.A.nranks
    sg = sigma if sigma is not None else list(range(P))
    inv = [0] * P
    for t, r in enumerate(sg):
        inv[r] = t
    npt = oracle.NUMPY[w.dtype]
    hb = []
    for s in range(P):
        b = np.empty(OB.local_elems(s), dtype=npt)
        oracle.fill(w.dtype, b, w.seed, synth.stream(synth.ROLE_B, 0, s))
        hb.append(b)
    ha = []
    for r in range(P):
        a = np.empty(OA.local_elems(inv[r]), dtype=npt)
        oracle.fill(w.dtype, a, w.seed, synth.stream(synth.ROLE_A, 0, r))
        ha.append(a)
    M, N = it.A.nrows, it.A.ncols
    # bands of target rows handed out in order (wrapping around) until
    # target_s has passed
    band = max(1, min((M + threads - 1) // threads, (1 << 22) // max(1, N)))
    nbands = (M + band - 1) // band
    lock = threading.Lock()
    state = {"next": 0, "elems": 0}
    t0 = time.perf_counter()

    def worker():
        while time.perf_counter() - t0 < target_s:
            with lock:
                k = state["next"] % nbands
                state["next"] += 1
            r0 = k * band
            r1 = min(M, r0 + band)
            oracle.transform(w.dtype, it.op, it.alpha, it.beta, OA, ha, OB, hb, sigma, r0, r1)
            with lock:
                state["elems"] += (r1 - r0) * N

    pool = [threading.Thread(target=worker) for _ in range(threads)]
    for t in pool:
        t.start()
    for t in pool:
        t.join()
    dt = time.perf_counter() - t0
    elems = state["elems"]
    return {"value": round(elems * model_bytes_per_elem / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{elems} elements of A in pair 0 (bands of {band} target rows of {M}, handed out in order, "
                      f"{elems / (M * N):.2f} passes over the {M}x{N} matrix) in {dt:.1f} s by {threads} threads; "
                      f"same bytes-per-element model as the GPU figure",
            "cpu": _cpu_model(), "seconds": round(dt, 2)}


def relabel_report() -> dict:
    """Local volume kept by the identity, the exact and the greedy relabeling
    (the paper's matching, Section 6) on every workload, with solve times."""
    import numpy as np
    import torch
    import synth
    import paper_2106_06601_amd as C
    torch.cuda.set_device(0)
    out = {}
    for name in synth.WORKLOADS:
        w = synth.workload(name)
        LA = [C.layout_from_spec(it.A) for it in w.items]
        LB = [C.layout_from_spec(it.B) for it in w.items]
        t0 = time.perf_counter()
        V = sum(C.costa_volume_matrix(a, b, it.op) for a, b, it in zip(LA, LB, w.items))
        t_v = time.perf_counter() - t0
        total = int(V.sum())
        t0 = time.perf_counter()
        sig_e, kept_id, kept_e = C.costa_relabel(V)
        t_e = time.perf_counter() - t0
        t0 = time.perf_counter()
        sig_g, _, after_g = C.costa_relabel_cost(V, method="greedy")
        t_g = time.perf_counter() - t0
        kept_g = total - int(after_g)
        out[name] = {"P": int(V.shape[0]), "total_elems": total,
                     "local_identity": int(kept_id), "local_exact": int(kept_e), "local_greedy": kept_g,
                     "remote_reduction_exact_pct": round(100 * (kept_e - kept_id) / max(1, total - kept_id), 3),
                     "remote_reduction_greedy_pct": round(100 * (kept_g - kept_id) / max(1, total - kept_id), 3),
                     "greedy_gap_pct_of_exact_gain": round(100 * (kept_e - kept_g) / max(1, kept_e - kept_id), 3),
                     "volume_ms": round(t_v * 1e3, 3), "exact_ms": round(t_e * 1e3, 3), "greedy_ms": round(t_g * 1e3, 3)}
    return {"metric": "relabeling: local volume kept (identity / exact / greedy)", "unit": "elements",
            "data": "synthetic", "workloads": out}


def bench2_sweep() -> dict:
    """Section 7.2 as a volume-only workload: 10^5 x 10^5 matrix, 10 x 10
    process grid, row-major ranks initially and column-major finally, target
    blocks 10^4, source block size varied from 1 to 10^4.  Volume matrix on
    the device (separable path), exact relabeling on the host."""
    import numpy as np
    import torch
    import synth
    import paper_2106_06601_amd as C
    torch.cuda.set_device(0)
    n, p, tb = 100000, 10, 10000
    LA = C.layout_from_spec(synth.BlockCyclic(n, n, tb, tb, p, p, "col", "col"))
    rows = []
    for b in (1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, 2000, 3000, 4000, 5000, 6000, 7000, 8000, 9000, 10000):
        LB = C.layout_from_spec(synth.BlockCyclic(n, n, b, b, p, p, "row", "col"))
        C.costa_timing_enable(True)
        t0 = time.perf_counter()
        V = C.costa_volume_matrix(LA, LB, "N")
        t_call = time.perf_counter() - t0
        kt = C.costa_timing_read()["volume"]
        C.costa_timing_enable(False)
        t0 = time.perf_counter()
        sigma, kept_id, kept = C.costa_relabel(V)
        t_lap = time.perf_counter() - t0
        remote_before, remote_after = n * n - kept_id, n * n - kept
        rows.append({"source_block": b, "remote_before": int(remote_before), "remote_after": int(remote_after),
                     "reduction_pct": round(100.0 * (remote_before - remote_after) / max(1, remote_before), 3),
                     "volume_kernel_ms": round(kt["ms"], 4), "volume_call_ms": round(t_call * 1e3, 3),
                     "relabel_ms": round(t_lap * 1e3, 3)})
    return {"metric": "communication-volume reduction from relabeling (Section 7.2 sweep)", "unit": "percent",
            "data": "synthetic (volume only)", "matrix": [n, n], "grid": [p, p], "target_block": tb, "sweep": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="blocksize_change_16k")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=min(16, os.cpu_count() or 1),
                    help="threads of the CPU baseline (default: up to 16, the host share of one GPU)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="before warm-up, run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--relabel-report", action="store_true",
                    help="print the relabeling comparison of every workload instead of the throughput line")
    ap.add_argument("--scalapack", metavar="NAME",
                    choices=["pdgemr2d_16k", "pdtran_16k", "pztranc_8k", "pdgemr2d_scatter_16k"],
                    help="time a ScaLAPACK-style call through its C entry point instead of the default workload")
    ap.add_argument("--bench2-sweep", action="store_true",
                    help="print the volume-reduction sweep of the paper's relabeling benchmark")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be >= 1 and --warmup >= 0")
    if args.bench2_sweep:
        print(json.dumps(bench2_sweep()), flush=True)
        return
    if args.relabel_report:
        print(json.dumps(relabel_report()), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the transform's virtual ranks all live in "
              "one GPU's HBM and this build has no multi-GPU exchange", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2106_06601_amd as C

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.scalapack:
        print(json.dumps(scalapack_bench(args.scalapack, args)), flush=True)
        return
    torch.cuda.set_device(0)
    w = synth.workload(args.workload)
    P = w.items[0].A.nranks
    stream = torch.cuda.current_stream()
    dev = torch.device("cuda:0")
    td = {"f64": torch.float64, "c128": torch.complex128, "f32": torch.float32, "c64": torch.complex64}[w.dtype]
    LA = [C.layout_from_spec(it.A) for it in w.items]
    LB = [C.layout_from_spec(it.B) for it in w.items]

    t_plan0 = time.perf_counter()
    sigma = None
    if w.relabel:
        V = sum(C.costa_volume_matrix(a, b, it.op) for a, b, it in zip(LA, LB, w.items))
        sigma, kept_id, kept_sigma = C.costa_relabel(V)
    inv = list(range(P)) if sigma is None else [0] * P
    if sigma is not None:
        for t, r in enumerate(sigma):
            inv[r] = t
    A, B = [], []
    for k, it in enumerate(w.items):
        A.append([torch.empty(LA[k].local_elems(inv[r]), dtype=td, device=dev) for r in range(P)])
        B.append([torch.empty(LB[k].local_elems(s), dtype=td, device=dev) for s in range(P)])
        for s, t in enumerate(B[k]):
            if t.numel():
                synth.fill_device(w.dtype, t.data_ptr(), t.numel(), w.seed, synth.stream(synth.ROLE_B, k, s),
                                  stream.cuda_stream)
        for r, t in enumerate(A[k]):
            if t.numel():
                synth.fill_device(w.dtype, t.data_ptr(), t.numel(), w.seed, synth.stream(synth.ROLE_A, k, r),
                                  stream.cuda_stream)
    descs = [dict(op=it.op, alpha=it.alpha, beta=it.beta, A=LA[k], A_local=A[k], B=LB[k], B_local=B[k])
             for k, it in enumerate(w.items)]
    stats = C.costa_plan_stats(w.dtype, descs, sigma)

    def step():
        if len(descs) == 1:
            d = descs[0]
            C.costa_transform(w.dtype, d["op"], d["alpha"], d["beta"], d["A"], d["A_local"], d["B"], d["B_local"],
                              sigma, stream)
        else:
            C.costa_transform_batched(w.dtype, descs, sigma, stream)

    t_setup = time.perf_counter() - t_plan0
    m = measure(step, stats, w.name, args)
    cpu = None
    if not args.no_cpu_baseline and len(w.items) == 1:
        cpu = cpu_baseline(w, sigma, stats["model_bytes"] / stats["total_elems"], args.cpu_seconds,
                           max(1, args.cpu_threads))

    out = {
        "metric": METRIC, "value": m["value"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": m["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "pct_of_hbm_peak": round(100 * m["value"] / HBM_PEAK_GBS, 2),
        "config": describe(w),
        "ms_per_step_median": m["ms_per_step_median"], "ms_per_step_min": m["ms_per_step_min"],
        "model_bytes_per_step": stats["model_bytes"],
        "bytes_without_staging_per_step": stats["model_bytes"] - 2 * stats["message_bytes"],
        "local_fraction": round(stats["local_elems"] / stats["total_elems"], 6),
        "waves": m["kernels"].get("pack", {}).get("launches_per_step", 0), "plan_s": round(t_setup + m["first_step_s"], 3),
        "kernels": m["kernels"],
        "roofline": m["roofline"],
        "copy_ceiling": m["copy_ceiling"],
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def measure(step, stats: dict, workload: str, args) -> dict:
    """Warm-up, then `args.steps` timed steps: per-launch HIP events on the
    launch stream plus one event pair around all steps."""
    import torch
    import paper_2106_06601_amd as C
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    if args.copy_probe:
        src = torch.ones(args.copy_probe << 17, dtype=torch.float64, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    t0 = time.perf_counter()
    step()  # builds and uploads the plan
    torch.cuda.synchronize()
    first_step_s = time.perf_counter() - t0
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    C.costa_timing_enable(True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    kt = C.costa_timing_read()
    C.costa_timing_enable(False)
    gpu_ms = ev[0].elapsed_time(ev[-1])
    per_step = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    ms_per_step = max(gpu_ms, wall * 1e3) / args.steps
    value = stats["model_bytes"] / (ms_per_step * 1e-3) / 1e9

    per_kernel = {}
    for k in KINDS:
        d = kt[k]
        if d["launches"]:
            per_kernel[k] = {"launches_per_step": d["launches"] / args.steps,
                             "ms_per_launch": round(d["ms"] / d["launches"], 5),
                             "bytes_per_launch": d["bytes"] // d["launches"],
                             "GB_s": round(d["bytes"] / (d["ms"] * 1e-3) / 1e9, 1)}
    dominant = max(per_kernel, key=lambda k: kt[k]["ms"])
    dk = per_kernel[dominant]
    achieved = dk["GB_s"]
    traffic = load_traffic(workload, dominant, dk["launches_per_step"])
    roof = {"bound": "hbm", "kernel": dominant, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
            "bytes_per_launch": dk["bytes_per_launch"], "ms_per_launch": dk["ms_per_launch"]}
    return {"value": round(value, 1), "ms_per_step": round(ms_per_step, 4), "kernels": per_kernel,
            "roofline": roof, "first_step_s": first_step_s, "copy_ceiling": copy_ceiling(dev, stream),
            "ms_per_step_median": round(per_step[len(per_step) // 2], 4), "ms_per_step_min": round(per_step[0], 4)}


def copy_ceiling(dev, stream, mib: int = 1024, reps: int = 10):
    """Context beside the 8 TB/s peak (not a target): a plain device-to-device
    copy of `mib` MiB (torch's copy_), read + write bytes over its event time,
    after the timed steps.  None when the memory is not free."""
    import torch
    nbytes = mib << 20
    if torch.cuda.mem_get_info(dev)[0] < 2 * nbytes + (256 << 20):
        return None
    src = torch.ones(nbytes // 8, dtype=torch.float64, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    torch.cuda.empty_cache()
    return {"GB_s": round(2 * nbytes / (ms * 1e-3) / 1e9, 1), "bytes_per_copy": 2 * nbytes,
            "kind": f"device copy of {mib} MiB (torch copy_), read + write bytes"}


def scalapack_bench(name: str, args) -> dict:
    """Throughput of a ScaLAPACK-style call through its C entry point
    (costa_pdgemr2d, costa_pdtran or costa_pztranc): descriptor and submatrix
    layouts, plans and message buffers come from the library's caches."""
    import torch
    import synth
    import paper_2106_06601_amd as C
    torch.cuda.set_device(0)
    call = synth.scalapack_call(name)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    td = {"f64": torch.float64, "c128": torch.complex128, "f32": torch.float32, "c64": torch.complex64}[call.dtype]
    LA, LC = C.layout_from_spec(call.A), C.layout_from_spec(call.C)
    a = [torch.empty(LA.local_elems(q), dtype=td, device=dev) for q in range(call.A.nranks)]
    c = [torch.empty(LC.local_elems(q), dtype=td, device=dev) for q in range(call.C.nranks)]
    for q, t in enumerate(a):
        if t.numel():
            synth.fill_device(call.dtype, t.data_ptr(), t.numel(), synth.DEFAULT_SEED,
                              synth.stream(synth.ROLE_B, 0, q), stream.cuda_stream)
    for q, t in enumerate(c):
        if t.numel():
            synth.fill_device(call.dtype, t.data_ptr(), t.numel(), synth.DEFAULT_SEED,
                              synth.stream(synth.ROLE_A, 0, q), stream.cuda_stream)
    tr = call.routine != "gemr2d"
    op = {"gemr2d": "N", "tran": "T", "tranu": "T", "tranc": "C"}[call.routine]
    ra, ca = (call.n, call.m) if tr else (call.m, call.n)
    sub_a = LA.submatrix(call.ia - 1, call.ja - 1, ra, ca)
    sub_c = LC.submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
    alpha, beta = (1.0, 0.0) if not tr else (call.alpha, call.beta)
    stats = C.costa_plan_stats(call.dtype, [dict(op=op, alpha=alpha, beta=beta, A=sub_c, B=sub_a)])
    ga = (call.A.nprow, call.A.npcol, call.A.rank_order, call.A.world, call.A.rank_map)
    gc = (call.C.nprow, call.C.npcol, call.C.rank_order, call.C.world, call.C.rank_map)
    da, dc = call.A.desc(), call.C.desc()
    fn = {"gemr2d": None, "tran": C.costa_pdtran, "tranc": C.costa_pztranc, "tranu": C.costa_pztranu}[call.routine]

    def step():
        if fn is None:
            C.costa_pdgemr2d(call.m, call.n, a, call.ia, call.ja, da, ga, c, call.ic, call.jc, dc, gc, stream)
        else:
            fn(call.m, call.n, call.alpha, a, call.ia, call.ja, da, ga, call.beta, c, call.ic, call.jc, dc, gc,
               stream)

    m = measure(step, stats, name, args)

    def dsc(d):
        ranks = f"ranks {d.rank_map} of {d.nranks}" if d.rank_map is not None else f"{d.rank_order}-major ranks"
        return (f"{d.m}x{d.n} in {d.mb}x{d.nb} blocks on a {d.nprow}x{d.npcol} grid ({ranks}), "
                f"RSRC {d.rsrc} CSRC {d.csrc} LLD {d.lld}")
    return {"metric": METRIC, "value": m["value"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": m["ms_per_step"], "higher_is_better": True,
            "dtype": call.dtype, "data": "synthetic", "pct_of_hbm_peak": round(100 * m["value"] / HBM_PEAK_GBS, 2),
            "config": {"workload": name, "routine": "p" + {"f64": "d", "c128": "z"}[call.dtype] + call.routine,
                       "m": call.m, "n": call.n, "alpha": str(call.alpha), "beta": str(call.beta),
                       "source": dsc(call.A) + f", submatrix at ({call.ia}, {call.ja})",
                       "target": dsc(call.C) + f", submatrix at ({call.ic}, {call.jc})"},
            "ms_per_step_median": m["ms_per_step_median"], "ms_per_step_min": m["ms_per_step_min"],
            "model_bytes_per_step": stats["model_bytes"],
            "bytes_without_staging_per_step": stats["model_bytes"] - 2 * stats["message_bytes"],
            "local_fraction": round(stats["local_elems"] / stats["total_elems"], 6),
            "kernels": m["kernels"], "roofline": m["roofline"]}


if __name__ == "__main__":
    main()
