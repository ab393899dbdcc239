"""Host-side tests of the ScaLAPACK-compatible layer (no GPU): descriptor and
submatrix layouts against the oracle's storage map, argument checks, and a
CPU replay of the plans of pxgemr2d / pxtran calls against the oracle's
window transform (every element of the destination submatrix written once,
nothing else touched, bit-exact)."""
import numpy as np
import pytest

import oracle
import synth
from replay import _combine, _index

C = pytest.importorskip("paper_2106_06601_amd")
PACK, UNPACK, DIRECT = 0, 1, 2


def _random_desc(rng, nprow, npcol, pad=None, maxdim=60):
    m, n = int(rng.integers(0, maxdim)), int(rng.integers(0, maxdim))
    mb, nb = int(rng.integers(1, 12)), int(rng.integers(1, 12))
    rsrc, csrc = int(rng.integers(0, nprow)), int(rng.integers(0, npcol))
    lr = max(oracle.numroc(m, mb, p, rsrc, nprow) for p in range(nprow))
    lld = max(1, lr) + (int(rng.integers(0, 4)) if pad is None else pad)
    return synth.ScaLapack(m, n, mb, nb, rsrc, csrc, lld, nprow, npcol, "row" if rng.random() < 0.5 else "col")


def _window_elements_match(L, O, i0, j0):
    """Every element of the library layout L (a window at (i0, j0) of the
    oracle's layout O): owner and offset as the oracle's storage map."""
    info = C.costa_layout_info(L.handle)
    rows, cols = info["nrows"], info["ncols"]
    if rows == 0 or cols == 0:
        return
    # walk the library's blocks, which tile the window; their extents come
    # from the descriptor's block size (_set_extents)
    own = np.full((rows, cols), -1, np.int64)
    off = np.full((rows, cols), -1, np.int64)
    r0 = 0
    for bi in range(info["nbr"]):
        c0 = 0
        h = None
        for bj in range(info["nbc"]):
            o, boff, ld = C.costa_layout_block(L.handle, bi, bj)
            w = _EXTENTS[(L.handle, "col")][bj]
            h = _EXTENTS[(L.handle, "row")][bi]
            ii, jj = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
            own[r0:r0 + h, c0:c0 + w] = o
            off[r0:r0 + h, c0:c0 + w] = boff + ii + jj * ld  # column-major local matrices
            c0 += w
        assert c0 == cols
        r0 += h
    assert r0 == rows
    ii, jj = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    rank, want = O.locate((ii + i0).ravel(), (jj + j0).ravel())
    assert np.array_equal(own.ravel(), rank) and np.array_equal(off.ravel(), want)


_EXTENTS = {}


def _set_extents(L, spec, i0, j0, m, n):
    """Block extents of a window, from the descriptor's block size (the
    boundaries of the full matrix's blocks that fall inside the window)."""
    def ext(start, length, b):
        if length == 0:
            return []
        cuts = [0] + [k * b - start for k in range(start // b + 1, (start + length - 1) // b + 1)] + [length]
        return list(np.diff(cuts))
    _EXTENTS[(L.handle, "row")] = ext(i0, m, spec.mb)
    _EXTENTS[(L.handle, "col")] = ext(j0, n, spec.nb)


def test_descriptor_and_window_layouts_match_oracle():
    rng = np.random.default_rng(41)
    for _ in range(40):
        pr, pc = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        d = _random_desc(rng, pr, pc)
        L = C.layout_from_spec(d)
        O = oracle.OLayout(d)
        assert [L.local_elems(q) for q in range(d.nranks)] == [O.local_elems(q) for q in range(d.nranks)]
        _set_extents(L, d, 0, 0, d.m, d.n)
        _window_elements_match(L, O, 0, 0)
        for _ in range(3):
            m, n = int(rng.integers(0, d.m + 1)), int(rng.integers(0, d.n + 1))
            i0, j0 = int(rng.integers(0, d.m - m + 1)), int(rng.integers(0, d.n - n + 1))
            S = L.submatrix(i0, j0, m, n)
            _set_extents(S, d, i0, j0, m, n)
            _window_elements_match(S, O, i0, j0)
            # a window of a window is the window of the full matrix
            if m and n:
                a, b = int(rng.integers(0, m)), int(rng.integers(0, n))
                T = S.submatrix(a, b, m - a, n - b)
                _set_extents(T, d, i0 + a, j0 + b, m - a, n - b)
                _window_elements_match(T, O, i0 + a, j0 + b)
            # buffer a rank needs for the window: one past its last window element
            ii, jj = np.meshgrid(np.arange(i0, i0 + m), np.arange(j0, j0 + n), indexing="ij")
            rank, off = O.locate(ii.ravel(), jj.ravel())
            for q in range(d.nranks):
                sel = rank == q
                assert S.local_elems(q) == (int(off[sel].max()) + 1 if sel.any() else 0)


def test_general_window_keeps_storage():
    spec = synth.workload("cosma_complex_16k", "small").items[0].B
    L = C.layout_from_spec(spec)
    O = oracle.OLayout(spec)
    rng = np.random.default_rng(42)
    for _ in range(5):
        m, n = int(rng.integers(1, 300)), int(rng.integers(1, 300))
        i0, j0 = int(rng.integers(0, spec.nrows - m)), int(rng.integers(0, spec.ncols - n))
        S = L.submatrix(i0, j0, m, n)
        info = C.costa_layout_info(S.handle)
        rs = [0] + [x - i0 for x in spec.row_splits if i0 < x < i0 + m] + [m]
        cs = [0] + [x - j0 for x in spec.col_splits if j0 < x < j0 + n] + [n]
        assert (info["nbr"], info["nbc"]) == (len(rs) - 1, len(cs) - 1)
        for bi in range(len(rs) - 1):
            for bj in range(len(cs) - 1):
                rank, off = O.locate(np.array([i0 + rs[bi]]), np.array([j0 + cs[bj]]))
                o, boff, _ = C.costa_layout_block(S.handle, bi, bj)
                assert (o, boff) == (rank[0], off[0])


def _status(fn, *a, **kw):
    try:
        fn(*a, **kw)
    except C.CostaError as e:
        return e.status
    return C.SUCCESS


def test_descriptor_and_call_errors():
    g = (2, 2, "row")
    good = [1, 0, 10, 10, 2, 2, 0, 0, 6]  # process row 0 holds 6 of the 10 rows
    assert _status(C.costa_layout_create_scalapack, good, 2, 2) == C.SUCCESS
    assert _status(C.costa_layout_create_scalapack, [2] + good[1:], 2, 2) == C.NOT_SUPPORTED
    assert _status(C.costa_layout_create_scalapack, good[:6] + [2, 0, 6], 2, 2) == C.INVALID_VALUE  # RSRC
    assert _status(C.costa_layout_create_scalapack, good[:7] + [-1, 6], 2, 2) == C.INVALID_VALUE  # CSRC
    assert _status(C.costa_layout_create_scalapack, good[:8] + [5], 2, 2) == C.INVALID_VALUE  # LLD < 6 rows
    assert _status(C.costa_layout_create_scalapack, good[:4] + [0, 2, 0, 0, 6], 2, 2) == C.INVALID_VALUE
    L = C.Layout.scalapack(good, 2, 2)
    assert _status(L.submatrix, 5, 5, 6, 1) == C.INVALID_VALUE
    assert _status(L.submatrix, -1, 0, 1, 1) == C.INVALID_VALUE
    bufs = [0x1000] * 4
    # argument errors come back before any device work (none is available here)
    assert _status(C.costa_pdgemr2d, 4, 4, bufs, 0, 1, good, g, bufs, 1, 1, good, g, stream=0) == C.INVALID_VALUE
    assert _status(C.costa_pdgemr2d, 4, 4, bufs, 8, 1, good, g, bufs, 1, 1, good, g, stream=0) == C.INVALID_VALUE
    assert _status(C.costa_pdgemr2d, -1, 4, bufs, 1, 1, good, g, bufs, 1, 1, good, g, stream=0) == C.INVALID_VALUE
    assert _status(C.costa_pdgemr2d, 4, 4, bufs, 1, 1, good, g, bufs, 1, 1, good, (1, 2, "row"),
                   stream=0) == C.SHAPE_MISMATCH
    assert _status(C.costa_pxtran, "f64", "N", 4, 4, 1.0, bufs, 1, 1, good, g, 0.0, bufs, 1, 1, good, g,
                   stream=0) == C.INVALID_VALUE
    # quick return: nothing to do, nothing enqueued
    assert _status(C.costa_pdtran, 0, 4, 1.0, bufs, 1, 1, good, g, 0.0, bufs, 1, 1, good, g, stream=0) == C.SUCCESS


def _replay_call(call):
    """Plan of the library's transform for the call (the layouts its
    ScaLAPACK entry points build), replayed on host buffers, against the
    oracle's window transform."""
    tr = call.routine != "gemr2d"
    op = {"gemr2d": "N", "tran": "T", "tranu": "T", "tranc": "C"}[call.routine]
    alpha, beta = (1.0, 0.0) if not tr else (call.alpha, call.beta)
    ra, ca = (call.n, call.m) if tr else (call.m, call.n)
    LA = C.layout_from_spec(call.A).submatrix(call.ia - 1, call.ja - 1, ra, ca)
    LC = C.layout_from_spec(call.C).submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
    descs = [dict(op=op, alpha=alpha, beta=beta, A=LC, B=LA)]
    pieces = C.costa_plan_export(call.dtype, descs)
    stats = C.costa_plan_stats(call.dtype, descs)
    P = call.C.nranks
    npt = oracle.NUMPY[call.dtype]
    OA, OC = oracle.OLayout(call.A), oracle.OLayout(call.C)
    rng = np.random.default_rng(call.m * 1000 + call.n)

    def bufs(O):
        out = []
        for q in range(P):
            k = O.local_elems(q)
            v = rng.integers(-99, 99, size=k) / 16.0
            if call.dtype in ("c128", "c64"):
                v = v + 1j * rng.integers(-99, 99, size=k) / 16.0
            out.append(np.ascontiguousarray(v.astype(npt)))
        return out

    a_bufs, c_bufs = bufs(OA), bufs(OC)
    want = [c.copy() for c in c_bufs]
    oracle.scalapack_call(call, a_bufs, want)
    es = synth.ITEMSIZE[call.dtype]
    table = c_bufs + a_bufs + [np.full(stats["workspace_bytes"] // es, np.nan, dtype=npt)]
    hits = [np.zeros(c.size, np.int32) for c in c_bufs]
    for p in pieces:
        src, dst = _index(p)
        sb, db = table[p["src_buf"]], table[p["dst_buf"]]
        assert src.min() >= 0 and src.max() < sb.size and dst.min() >= 0 and dst.max() < db.size
        if p["kind"] == PACK:
            db[dst] = sb[src]
            continue
        a_old = db[dst] if complex(beta) != 0 else None
        db[dst] = _combine(call.dtype, sb[src], a_old, complex(alpha), complex(beta), op == "C")
        hits[p["dst_buf"]][dst] += 1
    ii, jj = np.meshgrid(np.arange(call.m) + call.ic - 1, np.arange(call.n) + call.jc - 1, indexing="ij")
    rank, off = OC.locate(ii.ravel(), jj.ravel())
    u = np.uint64 if call.dtype in ("f64", "c128") else np.uint32
    for q in range(P):
        expect_hits = np.zeros(c_bufs[q].size, np.int32)
        expect_hits[off[rank == q]] = 1
        assert np.array_equal(hits[q], expect_hits), f"rank {q}: window not written exactly once"
        assert np.array_equal(c_bufs[q].view(u), want[q].view(u)), f"rank {q} differs from the oracle"


@pytest.mark.parametrize("seed", range(16))
def test_replay_scalapack_calls(seed):
    rng = np.random.default_rng(100 + seed)
    routine = ["gemr2d", "tran", "tranu", "tranc"][seed % 4]
    dtype = ["f64", "c128", "f32", "c64"][(seed // 4) % 4]
    P = [4, 6, 2, 8][seed % 4]
    shapes = [(a, P // a) for a in range(1, P + 1) if P % a == 0]
    ga, gc = shapes[int(rng.integers(len(shapes)))], shapes[int(rng.integers(len(shapes)))]
    dA = _random_desc(rng, *ga, maxdim=90)
    dC = _random_desc(rng, *gc, maxdim=90)
    tr = routine != "gemr2d"
    mmax = min(dC.m, dA.n if tr else dA.m)
    nmax = min(dC.n, dA.m if tr else dA.n)
    m, n = int(rng.integers(1, mmax + 1)) if mmax else 0, int(rng.integers(1, nmax + 1)) if nmax else 0
    ra, ca = (n, m) if tr else (m, n)
    ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
    ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
    cplx = dtype in ("c128", "c64")
    alpha, beta = [(2 - 1j, 0.5), (1.0, 0.0), (0.5j, 1.0), (-1.0, 0.0)][seed % 4] if cplx else \
        [(2.0, 0.5), (1.0, 0.0), (-0.5, 1.0), (3.0, 0.0)][seed % 4]
    call = synth.ScaLapackCall(routine, dtype, m, n, alpha, beta, dA, ia, ja, dC, ic, jc)
    if m and n:
        _replay_call(call)


@pytest.mark.parametrize("name", synth.SCALAPACK_CALLS)
def test_full_size_scalapack_plans_stay_in_bounds(name):
    """Every rectangle of the full-size ScaLAPACK plans against the sizes of
    the full descriptors' local buffers (vectorised; no data)."""
    call = synth.scalapack_call(name)
    tr = call.routine != "gemr2d"
    op = {"gemr2d": "N", "tran": "T", "tranu": "T", "tranc": "C"}[call.routine]
    ra, ca = (call.n, call.m) if tr else (call.m, call.n)
    LA = C.layout_from_spec(call.A)
    LC = C.layout_from_spec(call.C)
    SA = LA.submatrix(call.ia - 1, call.ja - 1, ra, ca)
    SC = LC.submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
    descs = [dict(op=op, alpha=call.alpha, beta=call.beta, A=SC, B=SA)]
    x = C.costa_plan_export(call.dtype, descs)
    st = C.costa_plan_stats(call.dtype, descs)
    P = call.C.nranks
    OA, OC = oracle.OLayout(call.A), oracle.OLayout(call.C)
    sizes = np.zeros(2 * P + 1, np.int64)
    for q in range(P):
        sizes[q] = OC.local_elems(q)
        sizes[P + q] = OA.local_elems(q)
        assert SC.local_elems(q) <= sizes[q] and SA.local_elems(q) <= sizes[P + q]
    sizes[2 * P] = st["workspace_bytes"] // synth.ITEMSIZE[call.dtype]
    T = (x["flags"] & 1) == 1
    nx, ny = x["nx"].astype(np.int64), x["ny"].astype(np.int64)
    src_end = np.where(T, x["src_off"] + (nx - 1) * x["src_ld"] + ny - 1,
                       x["src_off"] + (ny - 1) * x["src_ld"] + nx - 1)
    dst_end = x["dst_off"] + (ny - 1) * x["dst_ld"] + nx - 1
    assert (x["src_off"] >= 0).all() and (x["dst_off"] >= 0).all()
    assert (src_end < sizes[x["src_buf"]]).all() and (dst_end < sizes[x["dst_buf"]]).all()
    assert (nx >= 1).all() and (ny >= 1).all() and ((ny == 1) | (x["dst_ld"] >= nx)).all()
    assert (nx * ny)[x["kind"] != PACK].sum() == st["total_elems"] == call.m * call.n


def _mapped(rng, d, world):
    d.world = world
    d.rank_map = [int(x) for x in rng.permutation(world)[:d.nprow * d.npcol]]
    return d


def test_rank_mapped_layouts_match_oracle():
    rng = np.random.default_rng(43)
    for _ in range(30):
        pr, pc = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        d = _mapped(rng, _random_desc(rng, pr, pc), int(rng.integers(pr * pc, pr * pc + 5)))
        L = C.layout_from_spec(d)
        O = oracle.OLayout(d)
        assert C.costa_layout_info(L.handle)["nranks"] == d.world
        assert [L.local_elems(q) for q in range(d.world)] == [O.local_elems(q) for q in range(d.world)]
        _set_extents(L, d, 0, 0, d.m, d.n)
        _window_elements_match(L, O, 0, 0)
        m, n = int(rng.integers(0, d.m + 1)), int(rng.integers(0, d.n + 1))
        i0, j0 = int(rng.integers(0, d.m - m + 1)), int(rng.integers(0, d.n - n + 1))
        S = L.submatrix(i0, j0, m, n)
        _set_extents(S, d, i0, j0, m, n)
        _window_elements_match(S, O, i0, j0)


def test_rank_map_errors():
    good = [1, 0, 10, 10, 2, 2, 0, 0, 6]
    assert _status(C.costa_layout_create_scalapack, good, 2, 2, "row", 6, [5, 0, 2, 3]) == C.SUCCESS
    assert _status(C.costa_layout_create_scalapack, good, 2, 2, "row", 6, [5, 0, 2, 6]) == C.INVALID_VALUE
    assert _status(C.costa_layout_create_scalapack, good, 2, 2, "row", 6, [5, 0, 5, 3]) == C.INVALID_VALUE
    assert _status(C.costa_layout_create_scalapack, good, 2, 2, "row", 3, [0, 1, 2, 3]) == C.INVALID_VALUE
    assert _status(C.costa_layout_create_scalapack, good, 2, 2, "row", 6) == C.INVALID_VALUE  # no map
    one = [1, 0, 10, 10, 2, 2, 0, 0, 10]
    bufs = [0x1000] * 6
    # grids over different numbers of ranks
    assert _status(C.costa_pdgemr2d, 4, 4, bufs, 1, 1, one, (1, 1, "row", 5, [0]), bufs, 1, 1, good,
                   (2, 2, "row", 6, [0, 1, 2, 3]), stream=0) == C.SHAPE_MISMATCH


@pytest.mark.parametrize("seed", range(12))
def test_replay_calls_between_grids_of_different_sizes(seed):
    """pxgemr2d / pxtran between grids of different shapes over one set of
    ranks: scatter from one process, gather to one process, and mixed grids."""
    rng = np.random.default_rng(300 + seed)
    routine = ["gemr2d", "tran", "tranc", "gemr2d"][seed % 4]
    dtype = ["f64", "c128"][(seed // 4) % 2]
    world = int(rng.integers(4, 9))
    pairs = [((1, 1), (2, 2)), ((2, 2), (1, 1)), ((1, 2), (2, 1)), ((2, 2), (1, 3)), ((1, 1), (1, 4))]
    ga, gc = pairs[seed % len(pairs)]
    dA = _mapped(rng, _random_desc(rng, *ga, maxdim=70), world)
    dC = _mapped(rng, _random_desc(rng, *gc, maxdim=70), world)
    tr = routine != "gemr2d"
    mmax, nmax = min(dC.m, dA.n if tr else dA.m), min(dC.n, dA.m if tr else dA.n)
    if mmax == 0 or nmax == 0:
        return
    m, n = int(rng.integers(1, mmax + 1)), int(rng.integers(1, nmax + 1))
    ra, ca = (n, m) if tr else (m, n)
    ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
    ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
    alpha, beta = (2 - 1j, 0.5) if dtype == "c128" else (2.0, 0.5)
    _replay_call(synth.ScaLapackCall(routine, dtype, m, n, alpha, beta, dA, ia, ja, dC, ic, jc))


@pytest.mark.parametrize("order", ["row", "col"])
def test_general_window_random_grids(order):
    """Windows of random general grids in either storage order: every element
    of the window keeps its owner and offset (oracle storage map)."""
    rng = np.random.default_rng(44 if order == "row" else 45)
    for _ in range(10):
        M, N, P = int(rng.integers(1, 80)), int(rng.integers(1, 80)), int(rng.integers(1, 6))
        nr, nc = int(rng.integers(1, min(M, 6) + 1)), int(rng.integers(1, min(N, 6) + 1))
        rs = [0] + sorted(rng.choice(np.arange(1, M), nr - 1, replace=False).tolist()) + [M] if nr > 1 else [0, M]
        cs = [0] + sorted(rng.choice(np.arange(1, N), nc - 1, replace=False).tolist()) + [N] if nc > 1 else [0, N]
        spec = synth.General(M, N, rs, cs, rng.integers(0, P, (len(rs) - 1) * (len(cs) - 1)).tolist(), P, order)
        L = C.layout_from_spec(spec)
        O = oracle.OLayout(spec)
        m, n = int(rng.integers(1, M + 1)), int(rng.integers(1, N + 1))
        i0, j0 = int(rng.integers(0, M - m + 1)), int(rng.integers(0, N - n + 1))
        S = L.submatrix(i0, j0, m, n)
        info = C.costa_layout_info(S.handle)
        wr = [0] + [x - i0 for x in rs if i0 < x < i0 + m] + [m]
        wc = [0] + [x - j0 for x in cs if j0 < x < j0 + n] + [n]
        assert (info["nbr"], info["nbc"], info["block_order"]) == (len(wr) - 1, len(wc) - 1, order)
        for bi in range(len(wr) - 1):
            for bj in range(len(wc) - 1):
                o, boff, ld = C.costa_layout_block(S.handle, bi, bj)
                h, w = wr[bi + 1] - wr[bi], wc[bj + 1] - wc[bj]
                ii, jj = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
                rank, off = O.locate((ii + i0 + wr[bi]).ravel(), (jj + j0 + wc[bj]).ravel())
                mine = boff + (ii * ld + jj if order == "row" else ii + jj * ld)
                assert (rank == o).all() and np.array_equal(off, mine.ravel())
