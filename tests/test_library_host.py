"""Host-side tests of the C-ABI library (no GPU needed): exported symbols,
argument validation, layouts against the oracle's independent storage maps,
the relabeling against the oracle's brute force / DP / exact solvers, and the
host planner's volumes against the oracle's volume matrix."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synth

C = pytest.importorskip("paper_2106_06601_amd")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BC, GEN = synth.BlockCyclic, synth.General


def test_every_declared_symbol_is_exported():
    header = open(os.path.join(ROOT, "include", "costa.h")).read()
    names = set(re.findall(r"^\s*(?:costa_status|const char\*)\s+(costa_\w+)\s*\(", header, re.M))
    assert len(names) == 28  # every entry point of the header
    lib = ctypes.CDLL(C.LIB_PATH)
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing


# ---------------------------------------------------------------------------
# validation (returns an error before any device work)
# ---------------------------------------------------------------------------
def _status(fn, *a):
    try:
        fn(*a)
    except C.CostaError as e:
        return e.status
    return C.SUCCESS


def test_layout_validation():
    mk = C.costa_layout_create
    assert _status(mk, 10, 10, [0, 5, 10], [0, 10], [0, 1], 2) == C.SUCCESS
    assert _status(mk, 10, 10, [0, 5, 5, 10], [0, 10], [0, 1, 0], 2) == C.INVALID_VALUE  # repeated split
    assert _status(mk, 10, 10, [0, 5, 9], [0, 10], [0, 1], 2) == C.INVALID_VALUE        # wrong end
    assert _status(mk, 10, 10, [1, 5, 10], [0, 10], [0, 1], 2) == C.INVALID_VALUE       # wrong start
    assert _status(mk, 10, 10, [0, 5, 10], [0, 10], [0, 2], 2) == C.INVALID_VALUE       # owner >= P
    assert _status(mk, 10, 10, [0, 5, 10], [0, 10], [0, -1], 2) == C.INVALID_VALUE      # owner < 0
    assert _status(mk, 10, 10, [0, 5, 10], [0, 10], [0, 1], 0) == C.INVALID_VALUE       # P = 0
    # explicit storage with a leading dimension smaller than the block
    assert _status(mk, 10, 10, [0, 10], [0, 10], [0], 1, "col", [0], [9]) == C.INVALID_VALUE
    assert _status(mk, 10, 10, [0, 10], [0, 10], [0], 1, "col", [0], [12]) == C.SUCCESS
    assert _status(mk, 0, 5, [0], [0, 5], [], 1) == C.SUCCESS                           # empty matrix
    bc = C.costa_layout_create_block_cyclic
    assert _status(bc, 10, 10, 0, 2, 1, 1) == C.INVALID_VALUE
    assert _status(bc, 10, 10, 2, 2, 0, 1) == C.INVALID_VALUE


def test_transform_argument_errors_before_device_work():
    A = C.Layout.block_cyclic(8, 6, 2, 2, 2, 1)
    B = C.Layout.block_cyclic(6, 8, 2, 2, 2, 1)
    Bbad = C.Layout.block_cyclic(8, 8, 2, 2, 2, 1)
    B3 = C.Layout.block_cyclic(6, 8, 2, 2, 3, 1)
    bufs = [1 << 20, 2 << 20]  # never dereferenced: every call below fails validation
    t = C.costa_transform
    assert _status(t, "f64", "N", 1.0, 0.0, A, bufs, B, bufs) == C.SHAPE_MISMATCH
    assert _status(t, "f64", "T", 1.0, 0.0, A, bufs, Bbad, bufs) == C.SHAPE_MISMATCH
    assert _status(t, "f64", "T", 1.0, 0.0, A, bufs, B3, bufs + [0]) == C.SHAPE_MISMATCH
    assert _status(t, "f64", "T", 1.0, 0.0, A, bufs, B, bufs, [0, 0]) == C.INVALID_VALUE   # not a permutation
    assert _status(t, "f64", "T", 1.0, 0.0, A, bufs, B, bufs, [0, 2]) == C.INVALID_VALUE
    assert _status(t, "f64", "T", 1.0, 0.0, A, [bufs[0], 0], B, bufs) == C.INVALID_VALUE  # null buffer
    lib = ctypes.CDLL(C.LIB_PATH)
    assert lib.costa_transform(7, 0, None, None, None, None, None, None, None, None) == C.INVALID_VALUE
    assert C.costa_status_string(C.SHAPE_MISMATCH) == "shape mismatch"


# ---------------------------------------------------------------------------
# layouts vs the oracle's storage maps
# ---------------------------------------------------------------------------
BC_CASES = [
    BC(37, 53, 4, 8, 3, 2, "row", "col"), BC(37, 53, 4, 8, 3, 2, "col", "row"),
    BC(10, 7, 3, 2, 4, 3, "row", "col"), BC(20000, 20000, 64, 64, 8, 4, "row", "col"),
    BC(20000, 20000, 100, 100, 4, 8, "row", "row"), BC(4096, 524288, 512, 512, 8, 8),
]


@pytest.mark.parametrize("spec", BC_CASES, ids=str)
def test_block_cyclic_storage_matches_oracle(spec):
    L = C.layout_from_spec(spec)
    O = oracle.OLayout(spec)
    for r in range(spec.nranks):
        assert L.local_elems(r) == O.local_elems(r)
    # first element of every block: same owner and offset as the oracle's formula
    bi = np.arange(L.nbr)
    bj = np.arange(L.nbc)
    rows = np.repeat(np.minimum(bi * spec.mb, spec.nrows - 1), len(bj))
    cols = np.tile(np.minimum(bj * spec.nb, spec.ncols - 1), len(bi))
    rank, off = O.locate(rows, cols)
    for k in range(0, rows.size, max(1, rows.size // 2000)):
        o, boff, _ = C.costa_layout_block(L.handle, int(rows[k] // spec.mb), int(cols[k] // spec.nb))
        assert (o, boff) == (rank[k], off[k])


def test_general_default_packing_matches_oracle():
    spec = synth.workload("cosma_complex_16k", "small").items[0].B
    L = C.layout_from_spec(spec)
    O = oracle.OLayout(spec)
    for r in range(spec.nranks):
        assert L.local_elems(r) == O.local_elems(r)
    rs, cs = spec.row_splits, spec.col_splits
    for bi in range(len(rs) - 1):
        for bj in range(len(cs) - 1):
            rank, off = O.locate(np.array([rs[bi]]), np.array([cs[bj]]))
            assert C.costa_layout_block(L.handle, bi, bj)[:2] == (rank[0], off[0])


# ---------------------------------------------------------------------------
# relabeling vs the oracle
# ---------------------------------------------------------------------------
def test_relabel_matches_oracle_with_ties():
    rng = np.random.default_rng(7)
    for P in list(range(1, 9)) * 3:
        V = rng.integers(0, 4, size=(P, P)).astype(np.int64)
        sig, r0, r1 = C.costa_relabel(V)
        assert sig == oracle.relabel_bruteforce(V)
        assert r0 == oracle.retained(V, list(range(P))) and r1 == oracle.retained(V, sig)
    for P in (11, 16):
        V = rng.integers(0, 6, size=(P, P)).astype(np.int64)
        assert C.costa_relabel(V)[0] == oracle.relabel_dp(V)


def test_relabel_large_random_and_structured():
    rng = np.random.default_rng(8)
    for P in (32, 64):
        V = rng.integers(0, 3, size=(P, P)).astype(np.int64) * 1000
        assert C.costa_relabel(V)[0] == oracle.relabel_exact(V)
    V = np.full((64, 64), 5, np.int64)
    assert C.costa_relabel(V)[0] == list(range(64))
    V = np.zeros((100, 100), np.int64)
    perm = rng.permutation(100)
    V[perm, np.arange(100)] = 10**8  # label t fed entirely by rank perm[t]
    assert C.costa_relabel(V)[0] == perm.tolist()


def test_relabel_errors():
    with pytest.raises(C.CostaError):
        C.costa_relabel(np.array([[1, -1], [0, 0]]))


# ---------------------------------------------------------------------------
# host planner vs the oracle's volume matrix
# ---------------------------------------------------------------------------
def _descs(w):
    keep, descs = [], []
    for it in w.items:
        a, b = C.layout_from_spec(it.A), C.layout_from_spec(it.B)
        keep += [a, b]
        descs.append(dict(op=it.op, alpha=it.alpha, beta=it.beta, A=a, B=b))
    return descs, keep


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_plan_volumes_match_oracle_small(name):
    w = synth.workload(name, "small")
    descs, keep = _descs(w)
    P = w.items[0].A.nranks
    V = sum(oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op) for it in w.items)
    sig = oracle.relabel(V) if w.relabel and P <= 16 else list(range(P))
    st = C.costa_plan_stats(w.dtype, descs, sig)
    es = synth.ITEMSIZE[w.dtype]
    total = sum(it.A.nrows * it.A.ncols for it in w.items)
    local = oracle.retained(V, sig)
    assert st["total_elems"] == total
    assert st["local_elems"] == local
    assert st["remote_elems"] == total - local
    reads_a = sum(it.A.nrows * it.A.ncols for it in w.items if it.beta != 0)
    assert st["model_bytes"] == es * (2 * total + reads_a + 2 * (total - local))


def test_plan_full_size_model_bytes():
    # closed-form byte counts of the full-size workloads (read B + read A if
    # beta != 0 + write A + 2 x message bytes)
    expect = {"reshuffle_transpose_1k": 29360128, "scaled_transpose_20k": 15799993856,
              "rpa_batched_tall_skinny": 667867414528}
    for name, mb in expect.items():
        w = synth.workload(name)
        descs, keep = _descs(w)
        assert C.costa_plan_stats(w.dtype, descs)["model_bytes"] == mb
    w = synth.workload("blocksize_change_16k")
    descs, keep = _descs(w)
    sig = [0, 2, 1, 3, 8, 10, 9, 11, 4, 6, 5, 7, 12, 14, 13, 15]
    st = C.costa_plan_stats(w.dtype, descs, sig)
    assert st["model_bytes"] == 7516192768 and st["local_elems"] == 67108864
    assert C.costa_plan_stats(w.dtype, descs)["model_bytes"] == 8321499136


def test_plan_waves_respect_workspace_limit():
    w = synth.workload("blocksize_change_16k", "small")
    descs, keep = _descs(w)
    try:
        C.costa_set_workspace_limit(1 << 20)
        st = C.costa_plan_stats(w.dtype, descs)
        assert st["waves"] >= 20 and st["workspace_bytes"] <= 1 << 20
    finally:
        C.costa_set_workspace_limit(0)
    st = C.costa_plan_stats(w.dtype, descs)
    assert st["waves"] == 1


@pytest.mark.spawns
def test_one_hip_runtime_whatever_the_import_order():
    """The binding, the seeded fill library and the C client library, loaded
    before anything imports torch, leave one HIP runtime in the process
    (torch's): two copies would each see a different set of devices."""
    import subprocess
    import sys
    code = """
import ctypes, os, sys
sys.path.insert(0, %r)
sys.path.insert(0, os.path.join(%r, "tests"))
import paper_2106_06601_amd
import synth
synth.lib()
from c_client import build_client
if os.path.exists(build_client.LIB_OUT):
    ctypes.CDLL(build_client.LIB_OUT)
import torch
maps = open("/proc/self/maps").read().splitlines()
print(len({l.split()[-1] for l in maps if "libamdhip64" in l}))
""" % (ROOT, ROOT)
    r = subprocess.run([sys.executable, "-c", code], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip().splitlines()[-1] == "1"


def test_noalloc_refuses_a_plan_whose_tables_exceed_its_scratch():
    """costa_transform_batched_noalloc plans before any device call: a plan
    whose tables pass its table area is refused with NOT_SUPPORTED, one that
    fits goes on to the device (here: none, so a device error).  The buffer
    addresses are never dereferenced: without a GPU nothing is launched."""
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("with a GPU present the fitting plan would launch its kernels")
    fake = lambda P: [4096 * (r + 1) for r in range(P)]  # noqa: E731
    for name, want in (("scaled_transpose_20k", C.NOT_SUPPORTED), ("blocksize_change_16k", C.DEVICE)):
        w = synth.workload(name)
        it = w.items[0]
        P = it.A.nranks
        d = dict(op=it.op, alpha=it.alpha, beta=it.beta, A=C.layout_from_spec(it.A), A_local=fake(P),
                 B=C.layout_from_spec(it.B), B_local=fake(P))
        assert _status(C.costa_transform_batched_noalloc, w.dtype, [d]) == want, name
        if want == C.NOT_SUPPORTED:
            assert "bytes of tables" in C.costa_last_error()


@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
def test_parallel_host_fill_equals_the_oracle_fill(dtype):
    """The chunked multi-threaded host fill (used for the CPU baseline's
    inputs) gives the generator's values, element for element."""
    n = 10007
    a = np.zeros(n, dtype=oracle.NUMPY[dtype])
    synth.fill_host_parallel(dtype, a, 99, synth.stream(synth.ROLE_A, 5, 3), threads=4, chunk=1000)
    b = np.zeros(n, dtype=oracle.NUMPY[dtype])
    oracle.fill(dtype, b, 99, synth.stream(synth.ROLE_A, 5, 3))
    assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
