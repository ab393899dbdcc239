"""bench.py's command-line contract: one GPU only, argument checks, and the
fields of the JSON line it prints."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _run(*args, timeout=300):
    return subprocess.run([sys.executable, BENCH, *args], cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                          text=True, timeout=timeout)


@pytest.mark.spawns
def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.spawns
def test_bad_step_counts_are_refused():
    assert _run("--steps", "0").returncode == 2
    assert _run("--warmup", "-1").returncode == 2


@pytest.mark.gpu
def test_json_line_has_the_contract_fields(monkeypatch, capsys):
    # in this process: a process that has used the GPU starts no other
    import bench
    import torch
    print("bench contract: reshuffle_transpose_1k, 5 steps", flush=True)
    capsys.readouterr()
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "reshuffle_transpose_1k", "--steps", "5",
                                      "--warmup", "2", "--cpu-seconds", "1"])
    bench.main()
    out = capsys.readouterr().out
    torch.cuda.empty_cache()
    lines = [l for l in out.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 2
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["vs_baseline"] is None and d["dtype"] == "f64" and d["data"] == "synthetic"
    assert d["config"]["workload"] == "reshuffle_transpose_1k"
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert "traffic" in roof
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["unit"] == "GB/s"
    assert cpu["sample"]
