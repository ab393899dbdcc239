"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bit-exact everywhere: the volume matrix and the relabeling (integers), pure
reshuffles and transposes, and the scaled cases too, since both sides round
every product and sum on its own (no FMA contraction).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from replay import long_stack_case, many_rank_cases, random_stack_case, short_walk_cases, stack_cases

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2106_06601_amd as C
    from parity import Case

BC, GEN = synth.BlockCyclic, synth.General


def _say(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------------------
# volume matrix and relabeling on device volumes
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_volume_matrix_small_matches_oracle(name):
    w = synth.workload(name, "small")
    _say(f"volume {name} small")
    for it in w.items:
        A, B = C.layout_from_spec(it.A), C.layout_from_spec(it.B)
        V = C.costa_volume_matrix(A, B, it.op)
        assert np.array_equal(V, oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op))


def test_volume_matrix_full_size_closed_forms():
    _say("volume full sizes")
    w = synth.workload("reshuffle_transpose_1k")
    it = w.items[0]
    V = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
    assert np.array_equal(V, oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op))
    assert C.costa_relabel(V)[0] == oracle.relabel_bruteforce(V)
    # 16384^2 block-size change: 64 non-zero pairs of 4,194,304; canonical sigma
    it = synth.workload("blocksize_change_16k").items[0]
    V = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
    assert (V == 4194304).sum() == 64 and V.sum() == 16384 * 16384
    assert C.costa_relabel(V)[0] == oracle.relabel_dp(V) == [0, 2, 1, 3, 8, 10, 9, 11, 4, 6, 5, 7, 12, 14, 13, 15]
    # 20000^2 scaled transpose: identity keeps 12,500,384 local
    it = synth.workload("scaled_transpose_20k").items[0]
    V = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
    assert V.sum() == 20000 * 20000 and np.trace(V) == 12500384
    # tall-skinny pairs: V = 4,194,304 where the closed form says so
    w = synth.workload("rpa_batched_tall_skinny")
    tot = np.zeros((64, 64), np.int64)
    for it in (w.items[0], w.items[4]):
        V = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
        s, t = np.meshgrid(np.arange(64), np.arange(64), indexing="ij")
        hit = (s // 8 == t % 8) if it.op == "N" else (s // 8 == t // 8)
        assert np.array_equal(V, np.where(hit, 4194304, 0))
        tot += 4 * V
    assert oracle.retained(tot, list(range(64))) == 1207959552


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_workload_small_full_compare(name):
    w = synth.workload(name, "small")
    _say(f"transform {name} small")
    case = Case(w)
    if w.relabel:
        V = sum(oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op) for it in w.items)
        assert np.array_equal(case.V, V)
        assert case.sigma == oracle.relabel(V)
    case.run()
    case.check_full()
    case.run() if w.items[0].beta == 0 else None  # a second call reuses the cached plan
    if w.items[0].beta == 0:
        case.check_full()


@pytest.mark.parametrize("name", ["reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k",
                                  "cosma_complex_16k"])
def test_workload_full_size_sampled(name):
    w = synth.workload(name)
    _say(f"transform {name} full size")
    beta0 = all(it.beta == 0 for it in w.items)
    case = Case(w, a_init="nan" if beta0 else "gen")
    if w.relabel:
        assert case.sigma == oracle.relabel(case.V)
    case.run()
    n = case.check_sampled()
    assert n > 100000
    if beta0:
        case.check_all_written()
    # every element of every rank, the oracle run on bands of rows on 16 host threads
    _say(f"transform {name} full size: every element")
    assert case.check_rows(0) == w.items[0].A.nrows * w.items[0].A.ncols
    case.free()


def test_workload_rpa_full_size_sampled():
    w = synth.workload("rpa_batched_tall_skinny")
    need = sum(2 * it.A.nrows * it.A.ncols * 8 for it in w.items)
    free, total = torch.cuda.mem_get_info()
    if free < need + (4 << 30):
        pytest.skip(f"needs {need / 2**30:.0f} GiB + workspace; {free / 2**30:.0f} GiB free")
    _say("transform rpa_batched_tall_skinny full size")
    case = Case(w)
    case.run()
    n = case.check_sampled(n_random=50000, n_corners=100000)
    assert n > 100000
    # every element of the eight ranks of process row 0 (target rows 0..511,
    # one block row of 512 x 524288, written by every wave) of an identity
    # pair and a transposed pair
    it = w.items[0]
    assert it.A.prow == 8 and it.A.mb == 512 and it.A.nrows == 4096 and it.A.rank_order == "row"
    for k in (0, 4):
        _say(f"transform rpa_batched_tall_skinny full size: every element of ranks 0-7 of pair {k}")
        assert w.items[k].op == ("N" if k == 0 else "T")
        assert case.check_rows(k, 0, 512, ranks=range(8)) == 512 * 524288
    case.free()


def test_launches_beyond_one_slice():
    """A launch of more than 2^23 workgroups runs in slices: two ranks swap the
    halves of a 69632^2 fp64 matrix (38.8 GB, 4.85e9 elements, every element
    remote: about 9.5 million workgroups per pack and unpack launch)."""
    M = N = 69632
    need = 3 * M * N * 8
    torch.cuda.empty_cache()
    free, total = torch.cuda.mem_get_info()
    if free < need + (8 << 30):
        pytest.skip(f"needs {need / 2**30:.0f} GiB; {free / 2**30:.0f} GiB free")
    A = GEN(M, N, [0, M], [0, N // 2, N], [0, 1], 2, "col")
    B = GEN(M, N, [0, M], [0, N // 2, N], [1, 0], 2, "col")
    w = synth.Workload("slices", "f64", [synth.Item(A, B, "N", 1.0, 0.0)], False, seed=77)
    descs = [dict(op="N", alpha=1.0, beta=0.0, A=C.layout_from_spec(A), B=C.layout_from_spec(B))]
    x = C.costa_plan_export("f64", descs)
    for kind in (0, 1):  # pack, unpack
        sel = x[x["kind"] == kind]
        assert int(sel["group"].max()) + 1 > 1 << 23
    _say("transform 69632^2 swap, two launch slices")
    case = Case(w, a_init="nan")
    case.run()
    assert case.check_sampled(n_random=100000, n_corners=100000) > 100000
    case.check_all_written()
    case.free()


# ---------------------------------------------------------------------------
# random layouts, every op / order / type / scalar combination
# ---------------------------------------------------------------------------
def _random_general(rng, M, N, P, order):
    nr = int(rng.integers(1, min(M, 9) + 1))
    nc = int(rng.integers(1, min(N, 9) + 1))
    rs = [0] + sorted(rng.choice(np.arange(1, M), nr - 1, replace=False).tolist()) + [M] if nr > 1 else [0, M]
    cs = [0] + sorted(rng.choice(np.arange(1, N), nc - 1, replace=False).tolist()) + [N] if nc > 1 else [0, N]
    owners = rng.integers(0, P, (len(rs) - 1) * (len(cs) - 1)).tolist()
    return GEN(M, N, rs, cs, owners, P, order)


def _random_layout(rng, M, N, P, order):
    if rng.random() < 0.5:
        for pr in range(1, P + 1):
            if P % pr == 0 and rng.random() < 0.5:
                break
        pr = pr if P % pr == 0 else 1
        return BC(M, N, int(rng.integers(1, 40)), int(rng.integers(1, 40)), pr, P // pr,
                  "row" if rng.random() < 0.5 else "col", order)
    return _random_general(rng, M, N, P, order)


SCALARS = [(1.0, 0.0), (2.0, 0.5), (-0.75, 1.25), (0.3, 0.0), (1.0, 1.0)]
CSCALARS = [(1.0, 0.0), (0.5 - 0.25j, 0.25 + 1j), (1 + 0j, 1 + 0j), (0.3 + 0.7j, 0.0)]


@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
def test_random_layouts_full_compare(dtype):
    rng = np.random.default_rng({"f64": 1, "c128": 2, "f32": 3, "c64": 4}[dtype])
    for case_no in range(24):
        P = int(rng.integers(1, 9))
        M, N = int(rng.integers(1, 300)), int(rng.integers(1, 300))
        op = ["N", "T", "C"][case_no % 3]
        oa = "col" if rng.random() < 0.5 else "row"
        ob = "col" if rng.random() < 0.5 else "row"
        A = _random_layout(rng, M, N, P, oa)
        B = _random_layout(rng, M if op == "N" else N, N if op == "N" else M, P, ob)
        sc = CSCALARS if dtype in ("c128", "c64") else SCALARS
        alpha, beta = sc[case_no % len(sc)]
        sigma = rng.permutation(P).tolist() if rng.random() < 0.5 else None
        w = synth.Workload(f"random{case_no}", dtype, [synth.Item(A, B, op, alpha, beta)], False, seed=case_no + 7)
        _say(f"random {dtype} case {case_no}: P={P} {M}x{N} op={op} A={A.kind}/{oa} B={B.kind}/{ob} "
             f"alpha={alpha} beta={beta} sigma={sigma}")
        case = Case(w, sigma=sigma)
        case.run()
        case.check_full()


@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
def test_random_larger_layouts_full_compare(dtype):
    """Random layouts large enough that rectangles span many tasks, several
    tile rows and columns, wide tasks and per-XCD ranges (up to 3000 x 3000,
    up to 16 ranks, block sizes 1-300), every element compared."""
    rng = np.random.default_rng({"f64": 21, "c128": 22, "f32": 23, "c64": 24}[dtype])
    for case_no in range(8 if dtype in ("f64", "c128") else 4):
        P = int(rng.integers(1, 17))
        M, N = int(rng.integers(500, 3001)), int(rng.integers(500, 3001))
        op = ["N", "T", "C"][case_no % 3]
        oa = "col" if rng.random() < 0.5 else "row"
        ob = "col" if rng.random() < 0.5 else "row"

        def lay(m, n, order):
            if rng.random() < 0.7:
                divs = [d for d in range(1, P + 1) if P % d == 0]
                pr = divs[int(rng.integers(0, len(divs)))]
                return BC(m, n, int(rng.integers(1, 301)), int(rng.integers(1, 301)), pr, P // pr,
                          "row" if rng.random() < 0.5 else "col", order)
            return _random_general(rng, m, n, P, order)

        A = lay(M, N, oa)
        B = lay(M if op == "N" else N, N if op == "N" else M, ob)
        sc = CSCALARS if dtype in ("c128", "c64") else SCALARS
        alpha, beta = sc[case_no % len(sc)]
        sigma = rng.permutation(P).tolist() if rng.random() < 0.5 else None
        w = synth.Workload(f"larger{case_no}", dtype, [synth.Item(A, B, op, alpha, beta)], False, seed=case_no + 70)
        _say(f"larger random {dtype} case {case_no}: P={P} {M}x{N} op={op} A={A.kind}/{oa} B={B.kind}/{ob} "
             f"alpha={alpha} beta={beta} sigma={sigma}")
        case = Case(w, sigma=sigma)
        case.run()
        case.check_full()
        case.free()


@pytest.mark.parametrize("k", [0, 1])
def test_many_virtual_ranks_full_compare(k):
    dtype, op, alpha, beta, A, B, sigma = many_rank_cases()[k]
    w = synth.Workload(f"many{k}", dtype, [synth.Item(A, B, op, alpha, beta)], sigma == "auto", seed=90 + k)
    _say(f"many ranks: P={A.nranks} {dtype} op={op} sigma={'relabel' if sigma == 'auto' else 'random'}")
    case = Case(w, sigma="auto" if sigma == "auto" else sigma)
    case.run()
    case.check_full()
    case.free()


def test_random_batched_full_compare():
    rng = np.random.default_rng(11)
    for case_no in range(6):
        P = int(rng.integers(1, 7))
        items = []
        for k in range(int(rng.integers(1, 5))):
            M, N = int(rng.integers(1, 200)), int(rng.integers(1, 200))
            op = ["N", "T"][int(rng.integers(0, 2))]
            A = _random_layout(rng, M, N, P, "col" if rng.random() < 0.5 else "row")
            B = _random_layout(rng, M if op == "N" else N, N if op == "N" else M, P,
                               "col" if rng.random() < 0.5 else "row")
            alpha, beta = SCALARS[int(rng.integers(0, len(SCALARS)))]
            items.append(synth.Item(A, B, op, alpha, beta))
        sigma = rng.permutation(P).tolist()
        w = synth.Workload(f"batch{case_no}", "f64", items, False, seed=100 + case_no)
        _say(f"batched case {case_no}: P={P} pairs={len(items)} sigma={sigma}")
        case = Case(w, sigma=sigma)
        case.run()
        case.check_full()


@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
def test_transposed_rectangles_around_the_tile_limits(dtype):
    """Transposed rectangles whose width and height sit on both sides of every
    LDS tile limit (one tile per rectangle, balanced tile columns, ragged edge
    tiles): W x H rectangles on the direct path (one rank) and through
    messages (two ranks that swap their blocks), with and without beta."""
    widths = [1, 2, 15, 16, 17, 63, 64, 65, 127, 128, 129, 200, 255, 256, 257, 300, 513]
    heights = [1, 3, 12, 13, 14, 16, 17, 18, 26, 27, 33, 34, 129]
    sc = CSCALARS if dtype in ("c128", "c64") else SCALARS
    k = 0
    for W in widths:
        for H in heights:
            op = "C" if dtype in ("c128", "c64") and k % 2 else "T"
            alpha, beta = sc[k % len(sc)]
            if k % 2:
                A = GEN(W, H, [0, W], [0, H], [0], 1, "col")
                B = GEN(H, W, [0, H], [0, W], [0], 1, "col")
            else:
                A = GEN(W, 2 * H, [0, W], [0, H, 2 * H], [0, 1], 2, "col")
                B = GEN(2 * H, W, [0, H, 2 * H], [0, W], [1, 0], 2, "col")
            _say(f"tile limits {dtype} W={W} H={H} op={op} alpha={alpha} beta={beta} ranks={A.nranks}")
            w = synth.Workload(f"tiles{k}", dtype, [synth.Item(A, B, op, alpha, beta)], False, seed=300 + k)
            case = Case(w)
            case.run()
            case.check_full()
            k += 1


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", range(5))
def test_short_row_walks_full_compare(k):
    """Row walks of 4-64 elements starting inside 128-byte lines (16-byte
    units and single elements, four element types, every arithmetic mode),
    every element compared."""
    w = short_walk_cases()[k]
    sigma = list(range(w.items[0].A.nranks))[::-1] if k == 1 else None
    it = w.items[0]
    _say(f"short walks {k}: {w.dtype} {it.A.nrows}x{it.A.ncols} op={it.op} sigma={sigma}")
    case = Case(w, sigma=sigma)
    case.run()
    case.check_full()


@pytest.mark.parametrize("k", range(5))
def test_stacked_walks_full_compare(k):
    """Row walks moved as stacks (rectangles that follow one another along a
    local column, on the source or the destination side; 16-byte units and
    single elements, four element types, copy, scale and axpby, a partly idle
    last wave, row counts off the wave task's rows), every element compared."""
    w = stack_cases()[k]
    it = w.items[0]
    _say(f"stacked walks {k}: {w.dtype} {it.A.nrows}x{it.A.ncols} alpha={it.alpha} beta={it.beta}")
    case = Case(w)
    case.run()
    case.check_full()


@pytest.mark.parametrize("seed", range(8))
def test_random_stacked_layouts_full_compare(seed):
    """Random ScaLAPACK-descriptor pairs whose walks stack (sizes, pads, first
    processes, all four element types; beta 0 and 0.5), every element
    compared."""
    w = random_stack_case(seed)
    it = w.items[0]
    _say(f"random stacked layouts {seed}: {w.dtype} {it.A.nrows}x{it.A.ncols} beta={it.beta}")
    case = Case(w)
    case.run()
    case.check_full()


def test_stacks_longer_than_the_limit_full_compare():
    """Stacks cut at 4096 rectangles (local columns of 70,000 rows in 16-row
    source blocks), every element compared."""
    w = long_stack_case()
    _say("long stacks: fp64 140000x3")
    case = Case(w)
    case.run()
    case.check_full()


def test_waves_with_tiny_workspace():
    _say("waves with a 256 KiB workspace")
    try:
        C.costa_set_workspace_limit(256 << 10)
        for name in ("blocksize_change_16k", "rpa_batched_tall_skinny", "cosma_complex_16k", "scaled_transpose_20k"):
            w = synth.workload(name, "small")
            descs = [dict(op=it.op, alpha=it.alpha, beta=it.beta, A=C.layout_from_spec(it.A),
                          B=C.layout_from_spec(it.B)) for it in w.items]
            assert C.costa_plan_stats(w.dtype, descs)["waves"] > 4
            case = Case(w)
            case.run()
            case.check_full()
    finally:
        C.costa_set_workspace_limit(0)


def test_degenerate_shapes():
    cases = [
        (GEN(1, 1, [0, 1], [0, 1], [0], 1, "col"), GEN(1, 1, [0, 1], [0, 1], [0], 1, "row"), "T"),
        (BC(1, 257, 1, 16, 1, 3, "row", "row"), BC(257, 1, 5, 1, 3, 1, "col", "col"), "T"),
        (BC(130, 1, 7, 1, 2, 1), BC(130, 1, 64, 1, 1, 2), "N"),
        (BC(5, 7, 100, 100, 2, 2), BC(7, 5, 3, 3, 2, 2), "C"),  # some ranks own nothing
    ]
    for k, (A, B, op) in enumerate(cases):
        for dtype in ("f64", "c128"):
            _say(f"degenerate case {k} {dtype}")
            w = synth.Workload(f"deg{k}", dtype, [synth.Item(A, B, op, 2.0, 0.5)], False, seed=k)
            case = Case(w)
            case.run()
            case.check_full()


def test_empty_matrix_is_a_no_op():
    A = C.Layout.general(0, 5, [0], [0, 5], [], 2)
    B = C.Layout.general(5, 0, [0, 5], [0], [], 2)
    C.costa_transform("f64", "T", 1.0, 0.0, A, [0, 0], B, [0, 0])
    torch.cuda.synchronize()


def test_unaligned_buffers_take_the_narrow_path():
    """Buffers offset by one element (8 bytes) are not 16-byte aligned."""
    it = synth.workload("blocksize_change_16k", "small").items[0]
    LA, LB = C.layout_from_spec(it.A), C.layout_from_spec(it.B)
    OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
    P = 16
    dA = [torch.zeros(OA.local_elems(r) + 1, dtype=torch.float64, device="cuda") for r in range(P)]
    dB = [torch.empty(OB.local_elems(s) + 1, dtype=torch.float64, device="cuda") for s in range(P)]
    hB = []
    for s in range(P):
        h = np.zeros(OB.local_elems(s))
        oracle.fill("f64", h, 5, synth.stream(synth.ROLE_B, 0, s))
        dB[s][1:].copy_(torch.from_numpy(h))
        hB.append(h)
    C.costa_transform("f64", "N", 1.0, 0.0, LA, [t[1:] for t in dA], LB, [t[1:] for t in dB])
    hA = [np.zeros(OA.local_elems(r)) for r in range(P)]
    oracle.transform("f64", "N", 1.0, 0.0, OA, hA, OB, hB)
    torch.cuda.synchronize()
    for r in range(P):
        assert np.array_equal(dA[r][1:].cpu().numpy(), hA[r])


def test_two_streams_share_the_workspace_safely():
    w = synth.workload("blocksize_change_16k", "small")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        c1 = Case(w, sigma=None)
    with torch.cuda.stream(s2):
        c2 = Case(w, sigma=None)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        c1.run()
    with torch.cuda.stream(s2):
        c2.run()
    torch.cuda.synchronize()
    c1.check_full()
    c2.check_full()


def test_host_threads_call_at_once():
    """Eight host threads call the library at the same moment (the binding
    releases the interpreter lock during each call), each with its own stream
    and buffers: four different plans, and one plan that four of the threads
    share (its first call builds it while the others wait on the library's
    lock).  Every element of every result compared."""
    import threading
    cases = []
    for name in ("reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k", "cosma_complex_16k"):
        with torch.cuda.stream(torch.cuda.Stream()):
            cases.append(Case(synth.workload(name, "small")))
    shared = synth.workload("rpa_batched_tall_skinny", "small")
    for _ in range(4):
        with torch.cuda.stream(torch.cuda.Stream()):
            cases.append(Case(shared))
    torch.cuda.synchronize()
    start = threading.Barrier(len(cases))
    errors = []

    def call(c):
        try:
            start.wait(timeout=60)
            c.run()
        except Exception as e:  # reported after the join
            errors.append(e)

    _say(f"{len(cases)} host threads call the library at once")
    threads = [threading.Thread(target=call, args=(c,)) for c in cases]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a call did not return"
    torch.cuda.synchronize()
    assert not errors, errors
    for c in cases:
        c.check_full()


@pytest.mark.parametrize("kind", ["messages", "direct_only"])
def test_one_plan_two_streams_different_buffers(kind):
    """Two calls of one cached plan with different buffers, on two streams,
    issued back to back while the first call's kernels still run (full
    16384^2 sizes): the second call's buffer table must not reach the first
    call's kernels.  direct_only: a plan without message buffers (the same
    layout for A and B), where nothing else orders the two calls."""
    if kind == "messages":
        w = synth.workload("blocksize_change_16k")
    else:
        L = BC(16384, 16384, 256, 256, 4, 4, "row", "col")
        w = synth.Workload("same_layout", "f64", [synth.Item(L, L, "N", 2.0, 0.5)], False, seed=33)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        c1 = Case(w, sigma=None)
    with torch.cuda.stream(s2):
        c2 = Case(w, sigma=None)
    torch.cuda.synchronize()
    _say(f"one plan, two streams: {kind}")
    with torch.cuda.stream(s1):
        c1.run()
    with torch.cuda.stream(s2):
        c2.run()
    torch.cuda.synchronize()
    c1.check_sampled(n_random=100000, n_corners=100000)
    c2.check_sampled(n_random=100000, n_corners=100000)
    c1.free()
    c2.free()


def test_timing_counters():
    w = synth.workload("blocksize_change_16k", "small")
    case = Case(w)
    C.costa_timing_enable(True)
    for _ in range(3):
        case.run()
    t = C.costa_timing_read()
    C.costa_timing_enable(False)
    # the direct rectangles ride in the unpack launch (no launch of their own)
    assert t["pack"]["launches"] == 3 and t["unpack"]["launches"] == 3 and t["direct"]["launches"] == 0
    assert t["pack"]["ms"] > 0
    descs = [dict(op=it.op, alpha=it.alpha, beta=it.beta, A=case.LA[0], B=case.LB[0]) for it in w.items]
    st = C.costa_plan_stats(w.dtype, descs, case.sigma)
    assert t["pack"]["bytes"] == 3 * st["pack_bytes"]
    assert t["unpack"]["bytes"] == 3 * (st["unpack_bytes"] + st["direct_bytes"])


# ---------------------------------------------------------------------------
# separable volume path and the Section 7.2 relabeling sweep
# ---------------------------------------------------------------------------
def _as_general(spec):
    """The same block-cyclic layout expressed as a general grid with explicit
    per-block storage (so costa_volume_matrix takes the general kernel)."""
    L = C.layout_from_spec(spec)
    nbr, nbc = L.nbr, L.nbc
    rs = np.minimum(np.arange(nbr + 1, dtype=np.int64) * spec.mb, spec.nrows)
    cs = np.minimum(np.arange(nbc + 1, dtype=np.int64) * spec.nb, spec.ncols)
    blocks = [C.costa_layout_block(L.handle, bi, bj) for bi in range(nbr) for bj in range(nbc)]
    owners = [b[0] for b in blocks]
    return C.Layout.general(spec.nrows, spec.ncols, rs, cs, owners, spec.nranks, spec.block_order,
                            [b[1] for b in blocks], [b[2] for b in blocks])


@pytest.mark.parametrize("name", ["reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k",
                                  "rpa_batched_tall_skinny"])
def test_separable_volume_equals_general_kernel(name):
    _say(f"separable vs general volume {name}")
    w = synth.workload(name, "small")
    for it in (w.items[0], w.items[-1]):
        V_sep = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
        V_gen = C.costa_volume_matrix(_as_general(it.A), _as_general(it.B), it.op)
        assert np.array_equal(V_sep, V_gen)
        assert np.array_equal(V_sep, oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op))


def test_bench2_sweep_volumes_and_relabeling():
    """Section 7.2: 10^5 x 10^5 on a 10 x 10 grid, row-major ranks initially,
    column-major finally, target blocks 10^4, source blocks varied.  Equal
    blocks: relabeling removes all remote volume (the paper's printed point)."""
    import json
    import os
    from scipy.optimize import linear_sum_assignment
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "bench2_equal_blocks.json")))
    n, p = g["matrix"][0], g["grid"][0]
    A = BC(n, n, g["target"]["block"], g["target"]["block"], p, p, g["target"]["rank_order"], "col")
    LA = C.layout_from_spec(A)
    for b in (10000, 5000, 3000, 1000, 7, 1):
        _say(f"sweep source block {b}")
        B = BC(n, n, b, b, p, p, g["source"]["rank_order"], "col")
        V = C.costa_volume_matrix(LA, C.layout_from_spec(B), "N")
        assert np.array_equal(V, oracle.volume_separable(A, B, "N"))
        sigma, kept_id, kept = C.costa_relabel(V)
        r, c = linear_sum_assignment(V.astype(np.float64), maximize=True)
        assert kept == int(V[r, c].sum())
        total = n * n
        reduction = 100.0 * (kept - kept_id) / (total - kept_id)
        if b == g["source"]["block"]:
            assert kept == total and round(reduction) == g["volume_reduction_percent"]
