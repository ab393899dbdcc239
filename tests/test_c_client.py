"""The C ABI used from C: a C99 program compiled against include/costa.h
(tests/c_client/costa_client.c) against the library and the Python binding.

CPU: the header compiles as C99 with -Wall -Wextra -Werror, and every result
of the host-only entry points printed by the C program (local sizes, plan
statistics, every field of every exported rectangle, relabelings, error
codes) equals what the binding reads through ctypes -- so the header, the
library and the binding agree on struct layouts and enum values.
GPU: the same C code, loaded as a library (the test process already uses
the GPU, so it starts no other process), runs a transform on buffers it
allocates with hipMalloc; the result equals the oracle's bit for bit.
"""
import ctypes
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
from c_client import build_client  # noqa: E402

C = pytest.importorskip("paper_2106_06601_amd")
BC = synth.BlockCyclic

# (A, B, op): A is M x N, B is op^-1 of it
CASES = [
    (BC(100, 70, 8, 16, 2, 3, "row", "col"), BC(70, 100, 5, 7, 3, 2, "col", "row"), "T"),
    (BC(64, 96, 16, 16, 2, 2, "row", "col"), BC(64, 96, 32, 8, 2, 2, "col", "col"), "N"),
    (BC(33, 47, 4, 5, 3, 1, "col", "row"), BC(47, 33, 6, 3, 1, 3, "row", "col"), "C"),
]


def _args(spec):
    return [str(spec.nrows), str(spec.ncols), str(spec.mb), str(spec.nb), str(spec.prow), str(spec.pcol),
            spec.rank_order[0], spec.block_order[0]]


def _checksum(x):
    h = 1469598103934665603
    mask = (1 << 64) - 1
    fields = ["kind", "wave", "group", "src_off", "dst_off", "src_ld", "dst_ld", "src_buf", "dst_buf", "nx", "ny",
              "item", "flags", "ntasks", "tile_x", "tile_y", "launch", "wide_group", "wide_ntasks"]
    for p in x:
        for f in fields:
            h = ((h ^ (int(p[f]) & mask)) * 1099511628211) & mask
    return h


@pytest.fixture(scope="module")
def fresh_client(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    return build_client.build(out=str(tmp_path_factory.mktemp("c_client") / "costa_client"))


@pytest.mark.parametrize("k", range(len(CASES)))
@pytest.mark.spawns
def test_c_program_agrees_with_the_binding(fresh_client, k):
    A, B, op = CASES[k]
    r = subprocess.run([fresh_client, "host", *_args(A), *_args(B), op], stdout=subprocess.PIPE,
                       stderr=subprocess.PIPE, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    lines = [l.split() for l in r.stdout.splitlines()]
    LA, LB = C.layout_from_spec(A), C.layout_from_spec(B)
    local = [l for l in lines if l[0] == "local"]
    assert [(int(a), int(b)) for _, _, a, b in local] == [(LA.local_elems(q), LB.local_elems(q))
                                                          for q in range(A.nranks)]
    descs = [dict(op=op, A=LA, B=LB)]
    st = C.costa_plan_stats("f64", descs)
    got = [int(v) for v in next(l for l in lines if l[0] == "stats")[1:]]
    names = ["total_elems", "local_elems", "remote_elems", "model_bytes", "message_bytes", "workspace_bytes",
             "overlay_blocks", "pack_bytes", "unpack_bytes", "direct_bytes", "waves", "pieces_pack",
             "pieces_unpack", "pieces_direct"]
    assert got == [int(st[n]) for n in names]
    x = C.costa_plan_export("f64", descs)
    cnt, h = next(l for l in lines if l[0] == "pieces")[1:]
    assert int(cnt) == len(x) and int(h) == _checksum(x)
    V = np.array([[0, 0, 0], [5, 0, 4], [4, 0, 0]], np.int64)
    sig, kept_id, kept = C.costa_relabel(V)
    assert next(l for l in lines if l[0] == "relabel")[1:] == [str(v) for v in [*sig, kept_id, kept]]
    sig, before, after = C.costa_relabel_cost(V, method="greedy")
    assert next(l for l in lines if l[0] == "greedy")[1:] == [*map(str, sig), f"{before:.1f}", f"{after:.1f}"]
    errors = [l[1:] for l in lines if l[0] == "error"]
    assert errors == [[str(C.INVALID_VALUE), "1"], [str(C.INVALID_VALUE)]]


@pytest.mark.gpu
@pytest.mark.parametrize("k", range(len(CASES)))
def test_c_program_transform_matches_oracle(tmp_path, k):
    lib = build_client.LIB_OUT
    assert os.path.exists(lib), "tests/c_client/libcosta_client.so is not built: run __graft_entry__.build()"
    client = ctypes.CDLL(lib)
    client.costa_client_gpu.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_char_p),
                                        ctypes.POINTER(ctypes.c_char_p), ctypes.c_char_p, ctypes.c_double,
                                        ctypes.c_double]
    A, B, op = CASES[k]
    alpha, beta = (2.0, 0.5) if k != 1 else (1.0, 0.0)
    OA, OB = oracle.OLayout(A), oracle.OLayout(B)
    P = A.nranks
    hb = []
    for s in range(P):
        b = np.zeros(OB.local_elems(s))
        oracle.fill("f64", b, 7, synth.stream(synth.ROLE_B, 0, s))
        hb.append(b)
    ha = []
    for q in range(P):
        a = np.zeros(OA.local_elems(q))
        oracle.fill("f64", a, 7, synth.stream(synth.ROLE_A, 0, q))
        ha.append(a)
    np.concatenate(hb).tofile(tmp_path / "b.bin")
    np.concatenate(ha).tofile(tmp_path / "a.bin")
    print(f"C client transform case {k}: P={P} op={op}", flush=True)
    argv = lambda spec: (ctypes.c_char_p * 8)(*[a.encode() for a in _args(spec)])
    rc = client.costa_client_gpu(str(tmp_path).encode(), argv(A), argv(B), op.encode(), alpha, beta)
    assert rc == 0
    got = np.fromfile(tmp_path / "out.bin", dtype=np.float64)
    oracle.transform("f64", op, alpha, beta, OA, ha, OB, hb, None)
    exp = np.concatenate(ha)
    assert np.array_equal(got.view(np.uint64), exp.view(np.uint64))
