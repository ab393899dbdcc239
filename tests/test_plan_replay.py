"""CPU replay of the library's plans: the rectangles the kernels will process
are applied on host buffers with numpy, exactly as the kernels address them.

This checks, without a GPU, that (1) every read and write of every kernel stays
inside its buffer (the device buffers are sized by costa_layout_local_elems and
the message workspace by the plan), (2) every element of A is written exactly
once, (3) message blocks of one wave do not overlap, and (4) pack -> unpack and
the direct path together reproduce the oracle bit for bit.
"""
import numpy as np
import pytest

import oracle
import synth
from replay import _combine, _index, long_stack_case, many_rank_cases, random_stack_case, short_walk_cases, stack_cases

C = pytest.importorskip("paper_2106_06601_amd")

PACK, UNPACK, DIRECT = 0, 1, 2

# The task contract of the kernels: a transposed rectangle (flag 1) is moved
# by one workgroup per LDS tile (tile_x x tile_y elements; a tile is at most
# MAXX[es] wide and its tile_x rows of tile_y | 1 elements fit the LDS array
# of CAP[es] elements; a rectangle that fits is one tile, wider ones use as
# few tile columns as MAXX allows, and cut tiles are not far below the LDS
# array); a row walk by one
# workgroup per 256 units (16-byte vectors when flag 2 is set, else
# elements); a run of small row walks (each but the last flagged 16) by one
# workgroup for all of them.
# A stack (flag 32; 64: stacked on the destination side, else the source)
# is a run of row walks of one pair, vector width and height, each with rows
# of STACK_RUN[0] to STACK_RUN[1] bytes, that follow one another along x on
# that side; its first rectangle holds the stack's length in flags bits
# 16-31.  It is cut into wave tasks of 64 units of x by STACK_ROWS rows, and
# moved by ceil(wave tasks / 4) workgroups, in both task tables.
CAP = {4: 4224, 8: 2176, 16: 3328}
MAXX = {4: 128, 8: 128, 16: 256}
LANES, GROUP_UNITS, GROUP_PIECES, WIDE_UNITS = 256, 128, 8, 512
STACK_RUN, STACK_ROWS = (128, 512), 4


def _stacks(ps, es):
    """{index of a stack's first rectangle: (length, workgroups)} of one
    launch, after checking the stack contract."""
    out = {}
    k = 0
    while k < len(ps):
        fl = int(ps[k]["flags"])
        if not fl & 32:
            assert fl >> 16 == 0
            k += 1
            continue
        n = fl >> 16
        assert n >= 2 and k + n <= len(ps), "a stack starts with its length"
        side = "dst" if fl & 64 else "src"
        h = ps[k]
        for j in range(k, k + n):
            q = ps[j]
            qf = int(q["flags"])
            assert qf & 32 and (qf & 64) == (fl & 64) and (j == k or qf >> 16 == 0)
            assert not qf & (1 | 16) and (qf & 2) == (fl & 2)
            assert int(q["item"]) == int(h["item"]) and int(q["ny"]) == int(h["ny"])
            assert STACK_RUN[0] <= int(q["nx"]) * es <= STACK_RUN[1]
            if j > k:
                p = ps[j - 1]
                assert int(q[side + "_buf"]) == int(p[side + "_buf"])
                assert int(q[side + "_off"]) == int(p[side + "_off"]) + int(p["nx"]), "stacked rectangles are contiguous"
                assert int(h["ny"]) == 1 or int(q[side + "_ld"]) == int(p[side + "_ld"])
        width = sum(int(ps[j]["nx"]) for j in range(k, k + n)) // (16 // es if fl & 2 and es < 16 else 1)
        out[k] = (n, -(-(-(-width // 64) * -(-int(h["ny"]) // STACK_ROWS)) // (LANES // 64)))
        k += n
    return out


def check_tasks(pieces, es):
    """Every launch's workgroups are handed out in rectangle order without gaps
    or overlaps, each rectangle gets the number its tiles or units need, and
    runs of small rectangles fit one workgroup."""
    launches = {}
    for i, p in enumerate(pieces):
        launches.setdefault((int(p["kind"]), int(p["launch"])), []).append(p)
    order = [int(p["launch"]) for p in pieces]
    assert order == sorted(order), "rectangles are exported in launch order"
    for (kind, _), ps in launches.items():
        assert len({int(p["wave"]) for p in ps}) == 1 and len({int(p["kind"]) for p in ps}) == 1
        T = {bool(int(p["flags"]) & 1) for p in ps}
        assert kind == PACK and T == {False} or len(T) == 1, "a launch holds tiles or row walks, not both"
    for ps in launches.values():
        stacks = _stacks(ps, es)
        assert not stacks or not any(int(p["flags"]) & 1 for p in ps), "stacks only in launches of row walks"
        nxt = 0
        run = None  # (units so far, rectangles so far, item, vector width) of an open run
        skip = 0
        for i, p in enumerate(ps):
            if skip:
                skip -= 1
                continue
            if i in stacks:
                n, need = stacks[i]
                assert run is None
                for q in ps[i:i + n]:
                    assert int(q["group"]) == nxt and int(q["ntasks"]) == need
                nxt += need
                skip = n - 1
                continue
            nx, ny, fl = int(p["nx"]), int(p["ny"]), int(p["flags"])
            if run is not None:  # continues the run of the previous rectangle
                assert not fl & 1 and int(p["group"]) == nxt - 1 and int(p["ntasks"]) == 1
                units = nx * ny // (16 // es if fl & 2 and es < 16 else 1)
                assert units <= GROUP_UNITS and int(p["item"]) == run[2] and (fl & 2) == run[3]
                run = (run[0] + units, run[1] + 1, run[2], run[3])
                assert run[0] <= LANES and run[1] <= GROUP_PIECES
                if not fl & 16:
                    run = None
                continue
            assert int(p["group"]) == nxt, "workgroups of a launch are not handed out in order"
            if fl & 1:
                tx, ty = int(p["tile_x"]), int(p["tile_y"])
                assert 1 <= tx <= min(nx, MAXX[es]) and 1 <= ty <= ny and tx * (ty | 1) <= CAP[es]
                if nx <= MAXX[es] and nx * (ny | 1) <= CAP[es] - MAXX[es]:
                    assert (tx, ty) == (nx, ny), "a rectangle that fits a tile is one tile"
                if (tx, ty) != (nx, ny):
                    assert -(-nx // tx) == -(-nx // MAXX[es]), "more tile columns than needed"
                    assert ty == ny or 2 * tx * (ty + 2) > CAP[es] - MAXX[es], "tiles far below the LDS array"
                need = -(-nx // tx) * -(-ny // ty)
                assert not fl & 16
            else:
                units = nx * ny // (16 // es if fl & 2 and es < 16 else 1)
                need = -(-units // LANES)
                if fl & 16:
                    assert units <= GROUP_UNITS and need == 1
                    run = (units, 1, int(p["item"]), fl & 2)
            assert int(p["ntasks"]) == need, f"{p} needs {need} workgroups"
            nxt += need
        assert run is None, "a run of small rectangles ends with the launch's last rectangle flagged"
        # the wide task table of a launch of row walks: tasks of WIDE_UNITS
        # units, a run of small rectangles one task; none in launches with tiles
        if any(int(p["flags"]) & 1 for p in ps):
            assert all(int(p["wide_group"]) == -1 and int(p["wide_ntasks"]) == 0 for p in ps)
            continue
        nxt, in_run, skip = 0, False, 0
        for i, p in enumerate(ps):
            if skip:
                skip -= 1
                continue
            if i in stacks:
                n, need = stacks[i]
                for q in ps[i:i + n]:
                    assert int(q["wide_group"]) == nxt and int(q["wide_ntasks"]) == need
                nxt += need
                skip = n - 1
                continue
            nx, ny, fl = int(p["nx"]), int(p["ny"]), int(p["flags"])
            if in_run:
                assert int(p["wide_group"]) == nxt - 1 and int(p["wide_ntasks"]) == 1
                in_run = bool(fl & 16)
                continue
            assert int(p["wide_group"]) == nxt, "wide tasks of a launch are not handed out in order"
            units = nx * ny // (16 // es if fl & 2 and es < 16 else 1)
            need = 1 if fl & 16 else -(-units // WIDE_UNITS)
            assert int(p["wide_ntasks"]) == need
            in_run = bool(fl & 16)
            nxt += need


def _descs(w):
    keep, descs = [], []
    for it in w.items:
        a, b = C.layout_from_spec(it.A), C.layout_from_spec(it.B)
        keep += [a, b]
        descs.append(dict(op=it.op, alpha=it.alpha, beta=it.beta, A=a, B=b))
    return descs, keep


def _written_mask(it, sigma):
    """Per rank of A, the local elements that belong to the matrix (the
    oracle's transform of ones, marking what it writes; padding rows of a
    ScaLAPACK leading dimension stay 0)."""
    OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
    P = it.A.nranks
    sg = list(range(P)) if sigma is None else list(sigma)
    inv = [0] * P
    for t, r in enumerate(sg):
        inv[r] = t
    marks = [np.zeros(OA.local_elems(inv[r]), np.float64) for r in range(P)]
    ones = [np.ones(OB.local_elems(s), np.float64) for s in range(P)]
    oracle.transform("f64", "N" if it.op == "N" else "T", 1.0, 0.0, OA, marks, OB, ones, sigma)
    return [m.astype(np.int32) for m in marks]


def replay(w, sigma=None, limit=None, padded=False):
    """padded: A's local buffers hold elements outside the matrix (padded
    leading dimensions), which must stay unwritten."""
    descs, keep = _descs(w)
    if limit:
        C.costa_set_workspace_limit(limit)
    try:
        pieces = C.costa_plan_export(w.dtype, descs, sigma)
        stats = C.costa_plan_stats(w.dtype, descs, sigma)
    finally:
        if limit:
            C.costa_set_workspace_limit(0)
    n, P = len(w.items), w.items[0].A.nranks
    es = synth.ITEMSIZE[w.dtype]
    check_tasks(pieces, es)
    npt = oracle.NUMPY[w.dtype]
    sg = list(range(P)) if sigma is None else list(sigma)
    inv = [0] * P
    for t, r in enumerate(sg):
        inv[r] = t
    bufs = [None] * (2 * n * P + 1)
    hits = []
    for k, it in enumerate(w.items):
        OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
        for r in range(P):
            a = np.zeros(OA.local_elems(inv[r]), dtype=npt)
            oracle.fill(w.dtype, a, w.seed, synth.stream(synth.ROLE_A, k, r))
            bufs[k * P + r] = a
            hits.append(np.zeros(a.size, np.int32))
        for s in range(P):
            b = np.zeros(OB.local_elems(s), dtype=npt)
            oracle.fill(w.dtype, b, w.seed, synth.stream(synth.ROLE_B, k, s))
            bufs[n * P + k * P + s] = b
    msg_elems = stats["workspace_bytes"] // es
    bufs[2 * n * P] = np.full(msg_elems, np.nan, dtype=npt)
    # launch order as exported: DIRECT, then PACK/UNPACK per wave
    cur_wave, msg_used = -1, None
    for p in pieces:
        if p["kind"] == PACK and p["wave"] != cur_wave:
            cur_wave, msg_used = p["wave"], np.zeros(msg_elems, np.int8)
        src, dst = _index(p)
        sb, db = bufs[p["src_buf"]], bufs[p["dst_buf"]]
        assert src.min() >= 0 and src.max() < sb.size, f"read out of bounds in {p}"
        assert dst.min() >= 0 and dst.max() < db.size, f"write out of bounds in {p}"
        if p["kind"] == PACK:
            assert p["dst_buf"] == 2 * n * P and not (p["flags"] & 1)
            assert not msg_used[dst].any(), "message blocks overlap"
            msg_used[dst] = 1
            db[dst] = sb[src]
            continue
        it = w.items[p["item"]]
        alpha, beta = complex(it.alpha), complex(it.beta)
        a_old = db[dst] if beta != 0 else None
        db[dst] = _combine(w.dtype, sb[src], a_old, alpha, beta, it.op == "C")
        hits[p["dst_buf"]][dst] += 1
    # exactly once, and equal to the oracle
    for k, it in enumerate(w.items):
        OA, OB = oracle.OLayout(it.A), oracle.OLayout(it.B)
        ha = []
        for r in range(P):
            a = np.zeros(OA.local_elems(inv[r]), dtype=npt)
            oracle.fill(w.dtype, a, w.seed, synth.stream(synth.ROLE_A, k, r))
            ha.append(a)
        hb = [bufs[n * P + k * P + s] for s in range(P)]
        oracle.transform(w.dtype, it.op, it.alpha, it.beta, OA, ha, OB, hb, sigma)
        want = _written_mask(it, sigma) if padded else None
        for r in range(P):
            if padded:
                assert np.array_equal(hits[k * P + r], want[r]), "an element of A is not written exactly once"
                assert want[r].any() or want[r].size == 0
            else:
                assert np.all(hits[k * P + r] == 1), "an element of A is not written exactly once"
            u = np.uint64 if w.dtype in ("f64", "c128") else np.uint32
            assert np.array_equal(bufs[k * P + r].view(u), ha[r].view(u)), f"pair {k} rank {r} differs"
    return pieces, stats


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_replay_small_workloads(name):
    w = synth.workload(name, "small")
    sigma = None
    if w.relabel:
        V = sum(oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op) for it in w.items)
        sigma = oracle.relabel(V)
    replay(w, sigma)


def _waves_follow_receivers(pieces, P):
    """Plans of several waves take the packages receiver by receiver: the
    receivers of a wave's unpack rectangles (message sources) never come
    before those of the previous wave."""
    msg = pieces[(pieces["kind"] == UNPACK) & (pieces["src_buf"] == pieces["src_buf"].max())]
    last = -1
    for wv in np.unique(msg["wave"]):
        recv = msg["dst_buf"][msg["wave"] == wv] % P
        assert recv.min() >= last, "a wave takes packages of an earlier receiver"
        last = recv.max()


def test_replay_with_waves_and_relabeling():
    w = synth.workload("blocksize_change_16k", "small")
    pieces, stats = replay(w, sigma=[3, 1, 0, 2, 5, 4, 7, 6, 9, 8, 11, 10, 15, 12, 14, 13], limit=200 << 10)
    assert stats["waves"] > 10
    _waves_follow_receivers(pieces, 16)
    w = synth.workload("cosma_complex_16k", "small")
    pieces, stats = replay(w, limit=1 << 20)
    assert stats["waves"] > 1
    _waves_follow_receivers(pieces, 64)
    w = synth.workload("scaled_transpose_20k", "small")
    pieces, stats = replay(w, limit=4 << 20)
    assert stats["waves"] > 1
    _waves_follow_receivers(pieces, 32)


@pytest.mark.parametrize("seed", range(12))
def test_replay_random_layouts(seed):
    rng = np.random.default_rng(seed)
    BC, GEN = synth.BlockCyclic, synth.General
    P = int(rng.integers(1, 7))
    M, N = int(rng.integers(1, 150)), int(rng.integers(1, 150))
    op = ["N", "T", "C"][seed % 3]
    dtype = ["f64", "c128", "f32", "c64"][seed % 4]

    def lay(m, n, order):
        if rng.random() < 0.5:
            return BC(m, n, int(rng.integers(1, 20)), int(rng.integers(1, 20)), 1, P,
                      "row" if rng.random() < 0.5 else "col", order)
        nr, nc = int(rng.integers(1, min(m, 6) + 1)), int(rng.integers(1, min(n, 6) + 1))
        rs = [0] + sorted(rng.choice(np.arange(1, m), nr - 1, replace=False).tolist()) + [m] if nr > 1 else [0, m]
        cs = [0] + sorted(rng.choice(np.arange(1, n), nc - 1, replace=False).tolist()) + [n] if nc > 1 else [0, n]
        return GEN(m, n, rs, cs, rng.integers(0, P, (len(rs) - 1) * (len(cs) - 1)).tolist(), P, order)

    A = lay(M, N, "col" if rng.random() < 0.5 else "row")
    B = lay(M if op == "N" else N, N if op == "N" else M, "col" if rng.random() < 0.5 else "row")
    alpha, beta = [(1.0, 0.0), (2.0, 0.5), (0.5 - 0.25j, 0.25 + 1j)][seed % 3] if dtype in ("c128", "c64") \
        else [(1.0, 0.0), (2.0, 0.5), (-1.5, 0.0)][seed % 3]
    w = synth.Workload("r", dtype, [synth.Item(A, B, op, alpha, beta)], False, seed=seed)
    replay(w, sigma=rng.permutation(P).tolist())


@pytest.mark.parametrize("k", range(5))
def test_replay_short_row_walks(k):
    """Short misaligned row walks in every element type: in bounds, every
    element of A written once, equal to the oracle."""
    w = short_walk_cases()[k]
    pieces, _ = replay(w, sigma=list(range(w.items[0].A.nranks))[::-1] if k == 1 else None)
    assert not (pieces["flags"] & 1).any(), "the case has transposed rectangles"


@pytest.mark.parametrize("k", [0, 1])
def test_replay_many_virtual_ranks(k):
    """1024 and 4096 ranks, empty source process columns, relabeling by the
    library's exact LAP or a random permutation."""
    dtype, op, alpha, beta, A, B, sigma = many_rank_cases()[k]
    w = synth.Workload(f"many{k}", dtype, [synth.Item(A, B, op, alpha, beta)], sigma == "auto", seed=90 + k)
    if sigma == "auto":
        sigma = C.costa_relabel(oracle.volume(oracle.OLayout(A), oracle.OLayout(B), op))[0]
    replay(w, sigma=sigma)


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_full_size_plans_stay_in_bounds(name):
    """Every rectangle of the full-size plans against the buffer sizes
    (vectorised over rectangles; no data)."""
    w = synth.workload(name)
    descs, keep = _descs(w)
    P, n = w.items[0].A.nranks, len(w.items)
    sigma = None
    if name == "blocksize_change_16k":
        sigma = [0, 2, 1, 3, 8, 10, 9, 11, 4, 6, 5, 7, 12, 14, 13, 15]
    x = C.costa_plan_export(w.dtype, descs, sigma)
    st = C.costa_plan_stats(w.dtype, descs, sigma)
    es = synth.ITEMSIZE[w.dtype]
    sg = sigma or list(range(P))
    sizes = np.zeros(2 * n * P + 1, np.int64)
    for k, it in enumerate(w.items):
        for t in range(P):
            sizes[k * P + sg[t]] = C.costa_layout_local_elems(descs[k]["A"].handle, t)
            sizes[n * P + k * P + t] = C.costa_layout_local_elems(descs[k]["B"].handle, t)
    sizes[2 * n * P] = st["workspace_bytes"] // es
    T = (x["flags"] & 1) == 1
    nx, ny = x["nx"].astype(np.int64), x["ny"].astype(np.int64)
    src_end = np.where(T, x["src_off"] + (nx - 1) * x["src_ld"] + ny - 1,
                       x["src_off"] + (ny - 1) * x["src_ld"] + nx - 1)
    dst_end = x["dst_off"] + (ny - 1) * x["dst_ld"] + nx - 1
    assert (x["src_off"] >= 0).all() and (x["dst_off"] >= 0).all()
    assert (src_end < sizes[x["src_buf"]]).all()
    assert (dst_end < sizes[x["dst_buf"]]).all()
    assert (nx >= 1).all() and (ny >= 1).all() and (nx * ny <= 1 << 22).all()
    check_tasks(x, es)
    # rows of a rectangle do not wrap into each other
    assert ((ny == 1) | (x["dst_ld"] >= nx)).all()
    written = (nx * ny)[x["kind"] != PACK].sum()
    assert written == st["total_elems"]


def stack_walk_cover(ps, es):
    """The elements that the workgroups of each stack move, computed with the
    kernel's index arithmetic: wave v of task c takes wave task t = 4c + v
    (none past the stack's last), units [64 * (t % wb), +64) of x and rows
    [STACK_ROWS * (t // wb), +STACK_ROWS); the wave finds the last rectangle
    starting at or before its first unit by binary search, then scans forward
    while rectangles start before its end; each lane keeps the rectangle that
    holds its unit.  Returns {rectangle index: times each of its (y, x)
    elements is moved}."""
    cover = {}
    stacks = _stacks(ps, es)
    for k, (n, ntasks) in stacks.items():
        fl = int(ps[k]["flags"])
        side = "dst" if fl & 64 else "src"
        epu = 16 // es if fl & 2 and es < 16 else 1
        base = int(ps[k][side + "_off"])
        s0 = np.array([int(ps[j][side + "_off"]) - base for j in range(k, k + n)], np.int64)
        nxs = np.array([int(ps[j]["nx"]) for j in range(k, k + n)], np.int64)
        ny = int(ps[k]["ny"])
        hu = int((s0[-1] + nxs[-1]) // epu)
        wb = -(-hu // 64)
        nt = wb * -(-ny // STACK_ROWS)
        for j in range(n):
            cover[k + j] = np.zeros((ny, int(nxs[j])), np.int32)
        for c in range(ntasks):
            for v in range(LANES // 64):
                t = c * (LANES // 64) + v
                if t >= nt:
                    continue
                chunk, band = divmod(t, wb)
                y0, y1 = chunk * STACK_ROWS, min(chunk * STACK_ROWS + STACK_ROWS, ny)
                w0 = band * 64
                xw0, xw1 = w0 * epu, min(w0 + 64, hu) * epu
                lo, hi = 0, n - 1
                while lo < hi:
                    mid = (lo + hi + 1) >> 1
                    if s0[mid] <= xw0:
                        lo = mid
                    else:
                        hi = mid - 1
                xu = w0 + np.arange(64)
                x = xu * epu
                sel = np.full(64, -1)
                q = lo
                while q < n and s0[q] < xw1:
                    sel[(x >= s0[q]) & (x < s0[q] + nxs[q])] = q
                    q += 1
                for lane in np.nonzero(xu < hu)[0]:
                    q = sel[lane]
                    assert q >= 0, "a lane of the stack finds no rectangle"
                    xo = int(x[lane] - s0[q])
                    cover[k + q][y0:y1, xo:xo + epu] += 1
    return cover


@pytest.mark.parametrize("case", list(range(5)) + ["short_walks", "scaled_transpose_20k"])
def test_stack_walks_move_each_element_once(case):
    """The stack walk's lane arithmetic, replayed on the CPU over plans with
    stacks (and over cases whose walks do not stack): every element of every
    stacked rectangle is moved by exactly one lane of one workgroup."""
    if isinstance(case, int):
        ws = [stack_cases()[case]]
    elif case == "short_walks":
        ws = short_walk_cases()
    else:
        ws = [synth.workload(case, scale="small")]
    nstacked = 0
    for w in ws:
        descs, keep = _descs(w)
        x = C.costa_plan_export(w.dtype, descs, None)
        es = synth.ITEMSIZE[w.dtype]
        check_tasks(x, es)
        launches = {}
        for i in range(len(x)):
            launches.setdefault((int(x[i]["kind"]), int(x[i]["launch"])), []).append(x[i])
        for (kind, _), ps in launches.items():
            cover = stack_walk_cover(ps, es)
            nstacked += len(cover)
            if kind != PACK:  # outside the pack, stacks hold only pairs that do not read A
                assert all(complex(w.items[int(ps[k]["item"])].beta) == 0 for k in cover)
            for k, cv in cover.items():
                assert (cv == 1).all(), f"rectangle {k} of a stack: elements moved {cv.min()}..{cv.max()} times"
    if isinstance(case, int):
        assert nstacked > 0, "the case has no stacks"


@pytest.mark.parametrize("k", range(5))
def test_replay_stacked_walks(k):
    """Layouts whose walks stack, replayed rectangle by rectangle: in bounds,
    every element of A written once, equal to the oracle."""
    replay(stack_cases()[k], padded=True)


@pytest.mark.parametrize("name", ["scaled_transpose_20k", "rpa_batched_tall_skinny", "pdgemr2d_16k"])
def test_plans_do_not_depend_on_planner_threads(name, monkeypatch):
    """The planner's threads (pairs, ranges of strips, sorts and task tables
    split over up to 16) give the plan of a single thread, rectangle for
    rectangle and task for task (full sizes, where every split engages)."""
    import os
    if name in synth.WORKLOADS:
        w = synth.workload(name)
        descs, keep = _descs(w)
        dt = w.dtype
    else:
        call = synth.scalapack_call(name)
        SA = C.layout_from_spec(call.A).submatrix(call.ia - 1, call.ja - 1, call.m, call.n)
        SC = C.layout_from_spec(call.C).submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
        descs = [dict(op="N", alpha=1.0, beta=0.0, A=SC, B=SA)]
        dt = call.dtype
    limit = 18 << 30 if name == "rpa_batched_tall_skinny" else 0  # several waves
    out = {}
    for threads in ("1", "8"):
        monkeypatch.setenv("COSTA_PLAN_THREADS", threads)
        C.costa_finalize()  # empty the plan cache
        C.costa_set_workspace_limit(limit)
        try:
            out[threads] = (C.costa_plan_export(dt, descs, None), C.costa_plan_stats(dt, descs, None))
        finally:
            C.costa_set_workspace_limit(0)
    (x1, s1), (x8, s8) = out["1"], out["8"]
    assert len(x1) > 100000
    assert np.array_equal(x1.view(np.uint8), x8.view(np.uint8))
    for k in ("waves", "workspace_bytes", "pieces_pack", "pieces_unpack", "pieces_direct", "model_bytes"):
        assert s1[k] == s8[k], k


@pytest.mark.parametrize("seed", range(8))
def test_random_stacked_layouts(seed):
    """Random ScaLAPACK-descriptor pairs whose row walks stack: 2 x 2 grids,
    source blocks of 128-512 bytes of rows inside 128-row target blocks
    whose first process row is the other one, random sizes and padded
    leading dimensions (odd pads: single-element units), every element
    type, β = 0 (stacks on both sides) and β ≠ 0 (the pack's only):
    the stacks' lane arithmetic moves each element once, and the plan
    replayed rectangle by rectangle equals the oracle."""
    w = random_stack_case(seed)
    es = synth.ITEMSIZE[w.dtype]
    beta = complex(w.items[0].beta)
    descs, keep = _descs(w)
    x = C.costa_plan_export(w.dtype, descs, None)
    launches = {}
    for i in range(len(x)):
        launches.setdefault((int(x[i]["kind"]), int(x[i]["launch"])), []).append(x[i])
    nstacked = 0
    for (kind, _), ps in launches.items():
        for k, cv in stack_walk_cover(ps, es).items():
            nstacked += 1
            assert (cv == 1).all()
            if kind != PACK:
                assert beta == 0
    if beta == 0:
        assert nstacked > 0, "the case has no stacks"
    replay(w, padded=True)


def test_stacks_longer_than_the_limit_are_cut():
    """A local column of 4375 stackable rectangles: stacks of at most 4096,
    each element moved once, the plan equal to the oracle."""
    w = long_stack_case()
    descs, keep = _descs(w)
    x = C.costa_plan_export(w.dtype, descs, None)
    sizes = x["flags"] >> 16
    assert sizes.max() == 4096 and (sizes > 0).sum() >= 3
    launches = {}
    for i in range(len(x)):
        launches.setdefault((int(x[i]["kind"]), int(x[i]["launch"])), []).append(x[i])
    for ps in launches.values():
        for k, cv in stack_walk_cover(ps, 8).items():
            assert (cv == 1).all()
    replay(w, padded=True)
