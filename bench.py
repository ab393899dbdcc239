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
import gc
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


def host_cpus() -> dict:
    """What the host offers: logical CPUs of the machine, CPUs this process may
    run on, and the CPU model."""
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = os.cpu_count() or 1
    return {"nproc": os.cpu_count() or 1, "affinity": affinity, "cpu": _cpu_model()}


def cpu_baseline(w, sigma, model_bytes_per_elem: float, target_s: float, threads: int):
    """The CPU oracle on bands of target rows, run by `threads` threads at once
    (the oracle's C loop runs outside the GIL).  Pairs of a batch are taken one
    after another, each for an equal share of `target_s`, with only that pair's
    buffers in host memory; the figure is the elements of all pairs over the
    summed time."""
    import threading
    import numpy as np
    import oracle
    import synth
    P = w.items[0].A.nranks
    sg = sigma if sigma is not None else list(range(P))
    inv = [0] * P
    for t, r in enumerate(sg):
        inv[r] = t
    npt = oracle.NUMPY[w.dtype]
    per_item_s = target_s / len(w.items)
    total_elems, total_s, passes = 0, 0.0, []
    for k, it in enumerate(w.items):
        OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
        hb = []
        for s in range(P):
            b = np.empty(OB.local_elems(s), dtype=npt)
            synth.fill_host_parallel(w.dtype, b, w.seed, synth.stream(synth.ROLE_B, k, s), threads)
            hb.append(b)
        ha = []
        for r in range(P):
            a = np.empty(OA.local_elems(inv[r]), dtype=npt)
            synth.fill_host_parallel(w.dtype, a, w.seed, synth.stream(synth.ROLE_A, k, r), threads)
            ha.append(a)
        M, N = it.A.nrows, it.A.ncols
        # bands of target rows handed out in order (wrapping around) until
        # this pair's share of the time has passed
        band = max(1, min((M + threads - 1) // threads, (1 << 22) // max(1, N)))
        nbands = (M + band - 1) // band
        lock = threading.Lock()
        state = {"next": 0, "elems": 0}
        t0 = time.perf_counter()

        def worker():
            while time.perf_counter() - t0 < per_item_s:
                with lock:
                    b = state["next"] % nbands
                    state["next"] += 1
                r0 = b * band
                r1 = min(M, r0 + band)
                oracle.transform(w.dtype, it.op, it.alpha, it.beta, OA, ha, OB, hb, sigma, r0, r1)
                with lock:
                    state["elems"] += (r1 - r0) * N

        pool = [threading.Thread(target=worker) for _ in range(threads)]
        for t in pool:
            t.start()
        for t in pool:
            t.join()
        total_s += time.perf_counter() - t0
        total_elems += state["elems"]
        passes.append(state["elems"] / (M * N))
        del ha, hb
    it0 = w.items[0]
    what = (f"bands of target rows of the {it0.A.nrows}x{it0.A.ncols} matrix" if len(w.items) == 1 else
            f"each of the {len(w.items)} pairs in turn for {per_item_s:.1f} s, only its buffers in host memory; "
            f"bands of target rows of its {it0.A.nrows}x{it0.A.ncols} matrix")
    return {"value": round(total_elems * model_bytes_per_elem / total_s / 1e9, 4), "unit": "GB/s",
            "cores": threads, "kind": "oracle",
            "sample": f"{total_elems} elements of A ({what}, handed out in order; "
                      f"{', '.join(f'{p:.2f}' for p in passes)} passes over the matrix) in {total_s:.1f} s by "
                      f"{threads} threads; same bytes-per-element model as the GPU figure",
            "seconds": round(total_s, 2), **host_cpus()}


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
    # random layouts: two independent random general grids (random cuts, random
    # owners) of an 8192^2 matrix; greedy against exact under the locally-free
    # cost and under a two-level topology cost (nodes of 8 ranks)
    import numpy as np
    rand = []
    for P in (8, 16, 32, 64, 128, 256):
        rows = []
        for seed in range(5):
            A, B = synth.random_layout_pair(P, 1000 * P + seed, n=8192)
            V = C.costa_volume_matrix(C.layout_from_spec(A), C.layout_from_spec(B), "N")
            _, kept_id, kept_e = C.costa_relabel(V)
            _, _, after_g = C.costa_relabel_cost(V, method="greedy")
            kept_g = int(V.sum()) - int(after_g)
            node = np.arange(P) // 8
            same = node[:, None] == node[None, :]
            L = np.where(same, 0.0, 5.0)
            Bw = np.where(same, 1.0, 8.0)
            np.fill_diagonal(Bw, 0.0)
            _, w0, we = C.costa_relabel_cost(V, 8.0, L, Bw, "exact")
            _, _, wg = C.costa_relabel_cost(V, 8.0, L, Bw, "greedy")
            rows.append((kept_id, kept_e, kept_g, w0, we, wg))
        share = [100 * (g - i) / max(1, e - i) for i, e, g, *_ in rows]
        tshare = [100 * (w0 - wg) / (w0 - we) if w0 > we else 100.0 for *_, w0, we, wg in rows]
        rand.append({"P": P, "layouts": len(rows),
                     "local_identity_mean": round(float(np.mean([r[0] for r in rows])), 1),
                     "local_exact_mean": round(float(np.mean([r[1] for r in rows])), 1),
                     "local_greedy_mean": round(float(np.mean([r[2] for r in rows])), 1),
                     "greedy_share_of_exact_gain_pct": {"mean": round(float(np.mean(share)), 2),
                                                        "min": round(float(np.min(share)), 2)},
                     "topology_cost_reduction_exact_pct": round(float(np.mean([100 * (r[3] - r[4]) / r[3]
                                                                                for r in rows])), 2),
                     "topology_cost_reduction_greedy_pct": round(float(np.mean([100 * (r[3] - r[5]) / r[3]
                                                                                 for r in rows])), 2),
                     "topology_greedy_share_of_exact_gain_pct": {"mean": round(float(np.mean(tshare)), 2),
                                                                 "min": round(float(np.min(tshare)), 2)}})
    return {"metric": "relabeling: local volume kept (identity / exact / greedy)", "unit": "elements",
            "data": "synthetic", "workloads": out,
            "random_layouts": {"matrix": [8192, 8192], "source and target": "independent random general grids "
                               "(about 2 sqrt(P) random cuts per dimension, owners uniform over P)",
                               "topology": "nodes of 8 ranks: latency 0 and 1 unit/byte within a node, latency "
                                           "5 and 8 units/byte between nodes, 8-byte elements",
                               "rows": rand}}


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


# --------------------------------------------------------------------------
# profiles/: summaries of the rocprofv3 runs (the commands are in each file)
# --------------------------------------------------------------------------
PROFILE_WORKLOADS = ["reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k", "cosma_complex_16k",
                     "rpa_batched_tall_skinny"]
PROFILE_CALLS = ["pdgemr2d_16k", "pdgemr2d_scatter_16k", "pdtran_16k", "pztranc_8k"]
TRAFFIC_WORKLOADS = ["blocksize_change_16k", "scaled_transpose_20k", "cosma_complex_16k", "rpa_batched_tall_skinny",
                     "pdgemr2d_16k", "pdtran_16k", "pztranc_8k"]
LDS_WORKLOADS = ["reshuffle_transpose_1k", "cosma_complex_16k", "rpa_batched_tall_skinny", "pdtran_16k",
                 "pztranc_8k"]
PMC_READ = "TCC_BUBBLE_sum TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_32B_sum"
PMC_WRITE = "WRITE_SIZE TCC_EA0_RDREQ_DRAM_32B_sum TCC_EA0_WRREQ_WRITE_DRAM_32B_sum"
PMC_LDS = "SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE"
STALL_WORKLOADS = ["cosma_complex_16k", "blocksize_change_16k", "pztranc_8k"]
PMC_STALLS = ["SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_LDS SQ_INST_LEVEL_VMEM SQ_INSTS_VMEM "
              "SQ_ACTIVE_INST_VMEM",
              "TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum TCC_BUSY_sum GRBM_GUI_ACTIVE",
              "TA_BUSY_avr TA_ADDR_STALLED_BY_TC_CYCLES_sum GRBM_GUI_ACTIVE"]
_MODES = {0: "copy", 1: "scale", 2: "axpby", 3: "per pair"}
_TEMPLATE_NOTE = ("Kernel template arguments: <scalar, complex, kind (0 pack, 1 unpack-transform, 2 direct), "
                  "mode (0 copy, 1 scale, 2 axpby, 3 per pair), conjugate, LDS tiles>.")


def _bench_args(name: str) -> str:
    if name in PROFILE_CALLS:
        return f"--scalapack {name}"
    return f"--workload {name} --no-cpu-baseline --no-copy-ceiling"


def profile_commands(name: str, what: str) -> list:
    """The rocprofv3 commands behind a summary (run from /tmp with TMPDIR=/tmp;
    <out> is the directory given to --summarize-profiles, <repo> this tree)."""
    b = f"python3 <repo>/bench.py {_bench_args(name)}"
    if what == "trace":
        return [f"rocprofv3 --kernel-trace --stats -f csv -d <out>/trace_{name} -o run -- {b} --steps 20"]
    if what == "traffic":
        return [f"rocprofv3 --pmc {PMC_READ} -f csv -d <out>/pmcA_{name} -o run -- {b} --steps 2 --warmup 1 "
                f"--copy-probe 1024",
                f"rocprofv3 --pmc {PMC_WRITE} -f csv -d <out>/pmcB_{name} -o run -- {b} --steps 2 --warmup 1 "
                f"--copy-probe 1024"]
    if what == "stalls":
        return [f"rocprofv3 --pmc {c} -f csv -d <out>/stall{k}_{name} -o run -- {b} --steps 2 --warmup 1"
                for k, c in enumerate(PMC_STALLS)]
    return [f"rocprofv3 --pmc {PMC_LDS} -f csv -d <out>/lds_{name} -o run -- {b} --steps 2 --warmup 1"]


def _last_json(path: str) -> dict:
    with open(path) as fh:
        lines = [x for x in fh.read().splitlines() if x.startswith("{")]
    return json.loads(lines[-1])


def _short_name(name: str) -> str:
    n = name.strip()
    if n.startswith("void "):
        n = n[5:]
    depth, cut = 0, None
    for i in range(len(n) - 1, -1, -1):
        if n[i] == ")":
            depth += 1
        elif n[i] == "(":
            depth -= 1
            if depth == 0:
                cut = i
                break
    if cut is not None and n.endswith(")"):
        n = n[:cut]
    n = n.replace("costa::(anonymous namespace)::", "").replace("costa::", "").replace("(anonymous namespace)::", "")
    return n if len(n) <= 64 else n[:60]


def _mover_args(n: str):
    import re
    m = re.match(r"costa_mover(?:_lds)?<(\w+), (\w+), (\d), (\d), (\w+), (\w+)>", n)
    if not m:
        return None
    return {"kind": int(m.group(3)), "mode": int(m.group(4)), "conj": m.group(5) == "true",
            "tiles": m.group(6) == "true"}


def _role(n: str) -> str:
    a = _mover_args(n)
    if a:
        if a["kind"] == 0:
            return "pack"
        tags = [_MODES[a["mode"]]] + (["conjugate"] if a["conj"] else []) + (["LDS tiles"] if a["tiles"] else [])
        base = "unpack-transform (+direct rectangles)" if a["kind"] == 1 else "direct"
        return f"{base} [{', '.join(tags)}]"
    if "costa_volume" in n:
        return "volume matrix (planning, not timed)"
    if "copyBuffer" in n:
        return "plan/table upload or copy probe (setup)"
    if "fill_kernel" in n:
        return "seeded input fill (setup, not timed)"
    if n.startswith("at::"):
        return "torch (setup)"
    return "other"


def _pmc_values(path: str) -> dict:
    """{counter: {dispatch id: (kernel, value)}} of one --pmc run."""
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise RuntimeError(f"expected one counter_collection.csv under {path}, found {files}")
    out = {}
    with open(files[0]) as fh:
        for r in csv.DictReader(fh):
            key = r.get("Dispatch_Id") or r.get("Correlation_Id")
            d = out.setdefault(r["Counter_Name"], {})
            name, v = d.get(key, (r["Kernel_Name"], 0.0))
            d[key] = (name, v + float(r["Counter_Value"]))
    return out


def _per_kernel_mean(vals: dict) -> dict:
    """{short kernel name: (dispatches, mean value)} over the mover kernels."""
    acc = {}
    for name, v in vals.values():
        s = _short_name(name)
        if _mover_args(s) is None:
            continue
        a = acc.setdefault(s, [0, 0.0])
        a[0] += 1
        a[1] += v
    return {k: (n, tot / n) for k, (n, tot) in acc.items()}


def _probe_value(vals: dict) -> float:
    probes = [v for n, v in vals.values() if "copyBuffer" in n]
    if not probes:
        raise RuntimeError("no copy probe dispatch in the counter run")
    return max(probes)


def _title(name: str) -> str:
    if name in PROFILE_CALLS:
        return f"{name} (ScaLAPACK-style call through its C entry point)"
    import synth
    return f"{name} ({synth.workload(name).description})"


def summarize_profiles(src: str, out_dir: str = None) -> None:
    """Writes profiles/*.md (and the counters_*.json that bench.py reads for
    roofline.traffic) from the rocprofv3 output under `src`: whatever of
    trace_*, pmcA_*/pmcB_* and lds_* is there."""
    out_dir = out_dir or os.path.join(ROOT, "profiles")
    h = kernel_source_hash()
    stamp = f"Kernel source hash: `{h}` (bench.py's hash of the kernel, planner and launch sources)."
    wrote = []
    # kernel traces
    import csv
    import glob
    for name in PROFILE_WORKLOADS + PROFILE_CALLS:
        stats = glob.glob(os.path.join(src, f"trace_{name}", "**", "*kernel_stats.csv"), recursive=True)
        if not stats:
            continue
        d = _last_json(os.path.join(src, f"trace_{name}.json"))
        with open(stats[0]) as fh:
            rows = list(csv.DictReader(fh))
        lines = [f"# Kernel trace: {_title(name)}", "", "Command (from /tmp with TMPDIR=/tmp, on one MI355X):", "",
                 "```", *profile_commands(name, "trace"), "```", "",
                 "Each transform kernel: 1 plan-building call + 20 warm-up + 20 timed steps (times the launches per "
                 "step).", _TEMPLATE_NOTE, "",
                 "| kernel | role | calls | average (us) | min (us) | max (us) | share |",
                 "|---|---|---|---|---|---|---|"]
        for r in rows:
            n = _short_name(r["Name"])
            lines.append(f"| `{n}` | {_role(n)} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                         f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                         f"{float(r['Percentage']):.1f}% |")
        lines += ["", "Same kernels measured live by bench.py in the same run (HIP events around each launch on the "
                      "launch stream):", ""]
        for kind, k in d.get("kernels", {}).items():
            lines.append(f"- {kind}: {k['ms_per_launch'] * 1000:.1f} us per launch, {k['bytes_per_launch']} "
                         f"algorithmic bytes -> {k['GB_s']} GB/s ({k['launches_per_step']:g} launches per step)")
        lines.append(f"- whole step: {d['ms_per_step']} ms for {d['model_bytes_per_step']} model bytes -> "
                     f"{d['value']} GB/s ({d['pct_of_hbm_peak']}% of 8 TB/s)")
        r = d["roofline"]
        lines += [f"- roofline (dominant kernel {r['kernel']}): {r['achieved']} of {r['peak']:g} GB/s, "
                  f"frac {r['frac']}", "", stamp, ""]
        path = os.path.join(out_dir, f"kernel_trace_{name}.md")
        with open(path, "w") as fh:
            fh.write("\n".join(lines))
        wrote.append(path)
    # HBM traffic: FETCH_SIZE from its three inputs, WRITE_SIZE, and the
    # DRAM-side request counts, each calibrated on the 1 GiB device copy
    for name in TRAFFIC_WORKLOADS:
        pa, pb = os.path.join(src, f"pmcA_{name}"), os.path.join(src, f"pmcB_{name}")
        if not (os.path.isdir(pa) and os.path.isdir(pb)):
            continue
        A, B = _pmc_values(pa), _pmc_values(pb)
        dA = _last_json(os.path.join(src, f"pmcA_{name}.json"))

        def fetch_kib(bub, req, r32):
            return (bub * 128 + (req - bub - r32) * 64 + r32 * 32) / 1024

        # FETCH_SIZE per dispatch from its inputs
        fetch = {}
        for key, (kn, bub) in A["TCC_BUBBLE_sum"].items():
            req = A["TCC_EA0_RDREQ_sum"][key][1]
            r32 = A["TCC_EA0_RDREQ_32B_sum"][key][1]
            fetch[key] = (kn, fetch_kib(bub, req, r32))
        write = B["WRITE_SIZE"]
        dram_r = {k: (n, v * 32 / 1024) for k, (n, v) in B["TCC_EA0_RDREQ_DRAM_32B_sum"].items()}
        dram_w = {k: (n, v * 32 / 1024) for k, (n, v) in B["TCC_EA0_WRREQ_WRITE_DRAM_32B_sum"].items()}
        copy_kib = 1048576.0
        pf, pw = _probe_value(fetch), _probe_value(write)
        pdr, pdw = _probe_value(dram_r), _probe_value(dram_w)
        ff, wf, drf, dwf = copy_kib / pf, copy_kib / pw, copy_kib / pdr, copy_kib / pdw
        bub_share = {n: v for n, v in _per_kernel_mean(A["TCC_BUBBLE_sum"]).items()}
        req_share = _per_kernel_mean(A["TCC_EA0_RDREQ_sum"])
        r32_share = _per_kernel_mean(A["TCC_EA0_RDREQ_32B_sum"])
        F, W = _per_kernel_mean(fetch), _per_kernel_mean(write)
        DR, DW = _per_kernel_mean(dram_r), _per_kernel_mean(dram_w)
        pb_bub = _probe_value(A["TCC_BUBBLE_sum"])
        pb_req = _probe_value(A["TCC_EA0_RDREQ_sum"])
        pb_32 = _probe_value(A["TCC_EA0_RDREQ_32B_sum"])
        lines = [f"# HBM traffic counters: {_title(name)}", "",
                 "Commands (from /tmp with TMPDIR=/tmp; one rocprofv3 run per counter group):", "", "```",
                 *profile_commands(name, "traffic"), "```", "",
                 "FETCH_SIZE (KiB) = (TCC_BUBBLE x 128 + (TCC_EA0_RDREQ - TCC_BUBBLE - TCC_EA0_RDREQ_32B) x 64 + "
                 "TCC_EA0_RDREQ_32B x 32) / 1024, rocprofv3's gfx950 definition, computed here from its three "
                 "inputs; the DRAM counters count 32-byte units of the requests that go to memory (a 64-byte "
                 "request counts 2, a 128-byte one 4).", "",
                 f"Calibration on the plain device copy of 1024 MiB (`__amd_rocclr_copyBuffer`, `--copy-probe`): "
                 f"FETCH_SIZE {pf:.0f} KiB (TCC_BUBBLE {pb_bub:.0f}, TCC_EA0_RDREQ {pb_req:.0f}, 32-byte "
                 f"{pb_32:.0f}), WRITE_SIZE {pw:.0f} KiB, DRAM reads {pdr:.0f} KiB, DRAM writes {pdw:.0f} KiB, "
                 f"for 1048576 KiB moved each way: factors {ff:.5f} (fetch), {wf:.5f} (write), {drf:.5f} (DRAM "
                 f"read), {dwf:.5f} (DRAM write).", "",
                 "| kernel | role | dispatches | TCC_BUBBLE | TCC_EA0_RDREQ | RDREQ_32B | FETCH_SIZE (KiB) | "
                 "WRITE_SIZE (KiB) | DRAM read (KiB) | DRAM write (KiB) |",
                 "|---|---|---|---|---|---|---|---|---|---|"]
        kinds = {}
        for s in sorted(F):
            n, fv = F[s]
            wv, drv, dwv = W[s][1], DR[s][1], DW[s][1]
            lines.append(f"| `{s}` | {_role(s)} | {n} | {bub_share[s][1]:.0f} | {req_share[s][1]:.0f} | "
                         f"{r32_share[s][1]:.0f} | {fv:.0f} | {wv:.0f} | {drv:.0f} | {dwv:.0f} |")
            k = {0: "pack", 1: "unpack", 2: "direct"}[_mover_args(s)["kind"]]
            a = kinds.setdefault(k, [0, 0.0, 0.0, 0.0, 0.0])
            a[0] += n
            a[1] += fv * n
            a[2] += wv * n
            a[3] += drv * n
            a[4] += dwv * n
        lines += ["", "Per kernel kind (all launches of the kind; algorithmic bytes from bench.py's per-launch "
                      "figure of the same run; calibrated bytes = counter x 1024 x the copy's factor):", "",
                  "| kind | launches | FETCH+WRITE bytes per launch | ratio | DRAM read+write bytes per launch | "
                  "ratio | algorithmic bytes per launch |", "|---|---|---|---|---|---|---|"]
        for k, (n, sf, sw, sdr, sdw) in kinds.items():
            if k not in dA["kernels"]:  # launches the timed steps do not make
                continue
            hbm = round((sf / n * ff + sw / n * wf) * 1024)
            dram = round((sdr / n * drf + sdw / n * dwf) * 1024)
            alg = dA["kernels"][k]["bytes_per_launch"]
            lines.append(f"| {k} | {n} | {hbm} | {hbm / alg:.4f} | {dram} | {dram / alg:.4f} | {alg} |")
            with open(os.path.join(out_dir, f"counters_{k}_{name}.json"), "w") as fh:
                json.dump({"workload": name, "kernel": k, "kernel_source_hash": h, "fetch_kib": sf / n,
                           "write_kib": sw / n, "fetch_factor": ff, "write_factor": wf,
                           "dram_read_kib": sdr / n, "dram_write_kib": sdw / n, "dram_read_factor": drf,
                           "dram_write_factor": dwf, "hbm_bytes_per_launch": hbm, "dram_bytes_per_launch": dram,
                           "algorithmic_bytes_per_launch": alg}, fh, indent=1)
                fh.write("\n")
        lines += ["", "FETCH_SIZE and WRITE_SIZE count the L2's requests to the memory fabric; part of the fetches "
                      "can be served by the 256 MB Infinity Cache (MALL) behind it.  `roofline.traffic` in "
                      "bench.py's line is the FETCH+WRITE figure.", "", stamp, ""]
        path = os.path.join(out_dir, f"counters_traffic_{name}.md")
        with open(path, "w") as fh:
            fh.write("\n".join(lines))
        wrote.append(path)
    # LDS bank conflicts and occupancy (also of the odd-height tile variant)
    sections = []
    for prefix, name in [("lds", n) for n in LDS_WORKLOADS] + [("ldsodd", n) for n in LDS_WORKLOADS]:
        pl = os.path.join(src, f"{prefix}_{name}")
        if not os.path.isdir(pl):
            continue
        V = _pmc_values(pl)
        M = {c: _per_kernel_mean(V[c]) for c in PMC_LDS.split()}
        cmds = profile_commands(name, "lds")
        head = f"## {_title(name)}"
        if prefix == "ldsodd":
            head = f"## Variant with odd tile heights (COSTA_ODD_TILES=1): {_title(name)}"
            cmds = ["python3 <repo>/paper_2106_06601_amd/build.py --define COSTA_ODD_TILES=1 --out <lib>"] + \
                   [f"COSTA_LIB=<lib> {c.replace(f'lds_{name}', f'ldsodd_{name}')}" for c in cmds]
        sec = [head, "", "```", *cmds, "```", "",
               "| kernel | dispatches | SQ_INSTS_LDS | SQ_LDS_BANK_CONFLICT | conflicts per LDS instruction | "
               "SQ_WAVES | SQ_WAVE_CYCLES | GRBM_GUI_ACTIVE | resident waves per CU |",
               "|---|---|---|---|---|---|---|---|---|"]
        for s in sorted(M["SQ_WAVES"]):
            n = M["SQ_WAVES"][s][0]
            ins, conf = M["SQ_INSTS_LDS"][s][1], M["SQ_LDS_BANK_CONFLICT"][s][1]
            wc, gui = M["SQ_WAVE_CYCLES"][s][1], M["GRBM_GUI_ACTIVE"][s][1]
            per = f"{conf / ins:.3f}" if ins else "-"
            occ = 4 * wc / (gui / 8) / 256 if gui else 0.0
            sec.append(f"| `{s}` | {n} | {ins:.0f} | {conf:.0f} | {per} | {M['SQ_WAVES'][s][1]:.0f} | {wc:.4g} | "
                       f"{gui:.4g} | {occ:.1f} |")
        sections += sec + [""]
    if sections:
        lines = ["# LDS bank conflicts and occupancy", "",
                 "One rocprofv3 --pmc run per workload (from /tmp with TMPDIR=/tmp); counts are per dispatch (mean). "
                 "SQ_WAVE_CYCLES counts quad-cycles (4 clocks) and GRBM_GUI_ACTIVE is summed over the 8 XCDs "
                 "(about 8x the kernel's cycles); resident waves per CU = 4 x SQ_WAVE_CYCLES / (GRBM_GUI_ACTIVE / 8) "
                 "/ 256 CUs.", _TEMPLATE_NOTE, "", *sections, stamp, ""]
        path = os.path.join(out_dir, "counters_lds_occupancy.md")
        with open(path, "w") as fh:
            fh.write("\n".join(lines))
        wrote.append(path)
    # where the mover kernels wait: occupancy, time a vector memory
    # instruction stays outstanding, the address unit's stalls on the L1,
    # the L2's DRAM-credit stalls
    rows = []
    cmds = []
    for name in STALL_WORKLOADS:
        dirs = [os.path.join(src, f"stall{k}_{name}") for k in range(len(PMC_STALLS))]
        if not all(os.path.isdir(d) for d in dirs):
            continue
        cmds += profile_commands(name, "stalls")
        M = {}
        for d in dirs:
            for c, v in _pmc_values(d).items():
                M.setdefault(c, _per_kernel_mean(v))
        for k in sorted(M["SQ_WAVES"]):
            g = M["GRBM_GUI_ACTIVE"][k][1]
            occ = 4 * M["SQ_WAVE_CYCLES"][k][1] / (g / 8) / 256 if g else 0.0
            lvl = M["SQ_INST_LEVEL_VMEM"][k][1] / max(1.0, M["SQ_INSTS_VMEM"][k][1])
            ta = M["TA_ADDR_STALLED_BY_TC_CYCLES_sum"][k][1] / g if g else 0.0
            cr = (M["TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum"][k][1] + M["TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum"][k][1]) / g \
                if g else 0.0
            rows.append(f"| {name} | `{k}` | {_role(k)} | {occ:.1f} | {lvl:.1f} | {ta:.2f} | {cr:.3f} |")
    if rows:
        lines = ["# Where the mover kernels wait", "",
                 "Commands (from /tmp with TMPDIR=/tmp; one rocprofv3 run per counter set):", "", "```", *cmds, "```",
                 "", "Per dispatch, averaged over the dispatches of each kernel (the GRBM_GUI_ACTIVE of each run "
                     "normalises its own counters).  Resident waves per CU = 4 x SQ_WAVE_CYCLES / (GRBM_GUI_ACTIVE / "
                     "8 XCDs) / 256 CUs (SQ_WAVE_CYCLES counts quad-cycles; a CU holds 32 waves).  VMEM level = "
                     "SQ_INST_LEVEL_VMEM / SQ_INSTS_VMEM (how long a vector memory instruction stays "
                     "outstanding, relative).  TA address stalls on the vector L1 and the L2's DRAM-credit stalls "
                     "(reads + writes) per GRBM_GUI_ACTIVE cycle.", _TEMPLATE_NOTE, "",
                 "| workload | kernel | role | resident waves per CU | VMEM level | TA stalled by TC | "
                 "L2 DRAM-credit stalls |", "|---|---|---|---|---|---|---|", *rows, "", stamp, ""]
        path = os.path.join(out_dir, "counters_stalls_tiles_vs_walks.md")
        with open(path, "w") as fh:
            fh.write("\n".join(lines))
        wrote.append(path)
    for p in wrote:
        print("wrote", os.path.relpath(p, ROOT))


# The configurations the default run times, in this order: the block-size
# change first (the headline figure), the tall-skinny batch last (its 256 GiB
# of A and B need the device to themselves).
# the 1024^2 case first: launch-bound, its timed steps have shown one
# stall of tens of ms when they followed the block-size change's (and its
# device buffers' release) in the same process
ALL_WORKLOADS = ["reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k", "cosma_complex_16k",
                 "rpa_batched_tall_skinny"]
HEADLINE = "blocksize_change_16k"
NO_BANDWIDTH_CLAIM = {"reshuffle_transpose_1k": "29 MB per step, launch-bound and cache-resident: "
                                                "correctness case, no bandwidth claim"}


def run_workload(name: str, args, cpu_seconds: float) -> dict:
    """Plan, fill, time and (optionally) run the CPU baseline of one workload;
    frees its device memory and the library's plans before returning."""
    import torch
    import synth
    import paper_2106_06601_amd as C
    torch.cuda.set_device(0)
    w = synth.workload(name)
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
    # the device is no longer needed: free it before the CPU leg
    del A, B, descs, step
    torch.cuda.synchronize()
    C.costa_finalize()
    torch.cuda.empty_cache()
    cpu = None
    if cpu_seconds > 0:
        cpu = cpu_baseline(w, sigma, stats["model_bytes"] / stats["total_elems"], cpu_seconds,
                           max(1, args.cpu_threads))
    rec = {"value": m["value"], "unit": "GB/s", "ms_per_step": m["ms_per_step"],
           "pct_of_hbm_peak": round(100 * m["value"] / HBM_PEAK_GBS, 2), "dtype": w.dtype,
           "config": describe(w),
           "ms_per_step_median": m["ms_per_step_median"], "ms_per_step_min": m["ms_per_step_min"],
           "ms_per_step_max": m["ms_per_step_max"],
           "model_bytes_per_step": stats["model_bytes"],
           "bytes_without_staging_per_step": stats["model_bytes"] - 2 * stats["message_bytes"],
           "local_fraction": round(stats["local_elems"] / stats["total_elems"], 6),
           "waves": m["kernels"].get("pack", {}).get("launches_per_step", 0),
           "plan_s": round(t_setup + m["first_step_s"], 3),
           "kernels": m["kernels"], "roofline": m["roofline"], "cpu_baseline": cpu}
    if name in NO_BANDWIDTH_CLAIM:
        rec["note"] = NO_BANDWIDTH_CLAIM[name]
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="all", choices=["all"] + ALL_WORKLOADS,
                    help="one workload, or all of them (the headline figure is the block-size change; every "
                         "workload's figures are under 'configs')")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU-baseline time of a single workload (half of it per workload with 'all', 2 s for "
                         "the 1024^2 case)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", action="store_true",
                    help="skip the 1 GiB copy probes after the workloads (profiling runs: their launches would "
                         "join the kernel traces)")
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
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="write the profiles/ summaries from the rocprofv3 output under DIR (no GPU needed)")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be >= 1 and --warmup >= 0")
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles)
        return
    if args.bench2_sweep:
        print(json.dumps(bench2_sweep()), flush=True)
        return
    if args.relabel_report:
        print(json.dumps(relabel_report()), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the transform's virtual ranks all live in "
              "one GPU's HBM and the library has no multi-GPU exchange", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2106_06601_amd  # noqa: F401  (fails loudly when the library is not built)

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.scalapack:
        print(json.dumps(scalapack_bench(args.scalapack, args)), flush=True)
        return
    names = ALL_WORKLOADS if args.workload == "all" else [args.workload]
    recs = {}
    for name in names:
        if len(names) == 1:
            cs = args.cpu_seconds
        else:
            cs = 2.0 if name in NO_BANDWIDTH_CLAIM else args.cpu_seconds / 2
        if args.no_cpu_baseline:
            cs = 0.0
        print(f"bench: {name}", file=sys.stderr, flush=True)
        recs[name] = run_workload(name, args, cs)
    # context for the peak: a plain device copy, after every workload, so
    # that its 2 GiB of buffers are not allocated and freed between them
    head = recs[HEADLINE if HEADLINE in recs else names[0]]
    if not args.no_copy_ceiling:
        head["copy_ceiling"] = copy_ceiling(torch.device("cuda:0"), torch.cuda.current_stream())
    out = {"metric": METRIC, "value": head["value"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": head["ms_per_step"], "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": head["dtype"], "data": "synthetic",
           "pct_of_hbm_peak": head["pct_of_hbm_peak"], "config": head["config"]}
    for k in ("ms_per_step_median", "ms_per_step_min", "ms_per_step_max", "model_bytes_per_step",
              "bytes_without_staging_per_step",
              "local_fraction", "waves", "plan_s", "kernels", "roofline", "copy_ceiling", "cpu_baseline"):
        if k in head:
            out[k] = head[k]
    if len(names) > 1:
        claims = [r for n, r in recs.items() if n not in NO_BANDWIDTH_CLAIM]
        out["min_pct_of_hbm_peak"] = min(r["pct_of_hbm_peak"] for r in claims)
        out["min_roofline_frac"] = min(r["roofline"]["frac"] for r in claims)
        out["configs"] = recs
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
    # no garbage collection inside the timed steps: a full collection of the
    # objects earlier workloads left holds the host for tens of ms, long
    # enough for the GPU to run out of queued steps
    gc.collect()
    gc_was_on = gc.isenabled()
    gc.disable()
    try:
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        ev[0].record(stream)
        for i in range(args.steps):
            step()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
    finally:
        if gc_was_on:
            gc.enable()
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
            "roofline": roof, "first_step_s": first_step_s,
            "ms_per_step_median": round(per_step[len(per_step) // 2], 4), "ms_per_step_min": round(per_step[0], 4),
            "ms_per_step_max": round(per_step[-1], 4)}


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
    # the same copy through the library: an identity transform between two
    # single-rank layouts of one block (all of it on the direct path, the
    # row-walk kernel's plain copy)
    import synth
    import paper_2106_06601_amd as C
    n = nbytes // 8
    spec = synth.BlockCyclic(8192, n // 8192, 8192, n // 8192, 1, 1)
    L = C.layout_from_spec(spec)
    C.costa_transform("f64", "N", 1.0, 0.0, L, [dst], L, [src], None, stream)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        C.costa_transform("f64", "N", 1.0, 0.0, L, [dst], L, [src], None, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_costa = e0.elapsed_time(e1) / reps
    del src, dst, L
    C.costa_finalize()
    torch.cuda.empty_cache()
    return {"GB_s": round(2 * nbytes / (ms * 1e-3) / 1e9, 1), "bytes_per_copy": 2 * nbytes,
            "kind": f"device copy of {mib} MiB (torch copy_), read + write bytes",
            "costa_GB_s": round(2 * nbytes / (ms_costa * 1e-3) / 1e9, 1),
            "costa_kind": f"the same {mib} MiB through costa_transform (one rank, one block: the direct "
                          "path's row-walk copy)"}


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
            "ms_per_step_max": m["ms_per_step_max"],
            "model_bytes_per_step": stats["model_bytes"],
            "bytes_without_staging_per_step": stats["model_bytes"] - 2 * stats["message_bytes"],
            "local_fraction": round(stats["local_elems"] / stats["total_elems"], 6),
            "kernels": m["kernels"], "roofline": m["roofline"]}


if __name__ == "__main__":
    main()
