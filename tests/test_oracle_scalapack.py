"""Pins of the oracle's ScaLAPACK descriptors and windows (submatrices).

The oracle's storage map for a descriptor (first block on process row RSRC and
column CSRC, local leading dimension LLD) is checked against a simulation of
the dealing itself: blocks handed out one after another round the process
cycle, each process stacking what it receives.  Window transforms are checked
against numpy slicing of the gathered global matrices (Section 5: a submatrix
is taken by truncating the splits, so every element keeps its place)."""
import itertools

import numpy as np
import pytest

import oracle
import synth


def _deal(n, nb, nprocs, src):
    """(process, local index) of every index of an n-long dimension, by dealing
    nb-blocks round the cycle starting at process src."""
    proc = np.zeros(n, np.int64)
    local = np.zeros(n, np.int64)
    taken = [0] * nprocs
    p = src
    for start in range(0, n, nb):
        for g in range(start, min(n, start + nb)):
            proc[g] = p
            local[g] = taken[p]
            taken[p] += 1
        p = (p + 1) % nprocs
    return proc, local, taken


def _random_desc(rng, nprow=None, npcol=None, pad=None):
    nprow = nprow or int(rng.integers(1, 4))
    npcol = npcol or int(rng.integers(1, 4))
    m, n = int(rng.integers(0, 40)), int(rng.integers(0, 40))
    mb, nb = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    rsrc, csrc = int(rng.integers(0, nprow)), int(rng.integers(0, npcol))
    rows = _deal(m, mb, nprow, rsrc)[2]
    lld = max(1, max(rows)) + (int(rng.integers(0, 4)) if pad is None else pad)
    order = "row" if rng.random() < 0.5 else "col"
    return synth.ScaLapack(m, n, mb, nb, rsrc, csrc, lld, nprow, npcol, order)


def _rank(d, pr, pc):
    if d.rank_map is not None:
        return d.rank_map[pr + pc * d.nprow]
    return pr * d.npcol + pc if d.rank_order == "row" else pr + pc * d.nprow


def _brute_map(d):
    """rank[i, j] and offset[i, j] of every element by simulating the dealing."""
    pr, li, _ = _deal(d.m, d.mb, d.nprow, d.rsrc)
    pc, lj, _ = _deal(d.n, d.nb, d.npcol, d.csrc)
    rank = np.array([[_rank(d, a, b) for b in pc] for a in pr], np.int64).reshape(d.m, d.n)
    off = li[:, None] + lj[None, :] * d.lld
    return rank, off


def test_numroc_matches_dealing():
    rng = np.random.default_rng(31)
    for _ in range(300):
        n, nb, P = int(rng.integers(0, 200)), int(rng.integers(1, 20)), int(rng.integers(1, 9))
        src = int(rng.integers(0, P))
        taken = _deal(n, nb, P, src)[2]
        assert [oracle.numroc(n, nb, p, src, P) for p in range(P)] == taken


def test_descriptor_storage_map_matches_dealing():
    rng = np.random.default_rng(32)
    for _ in range(60):
        d = _random_desc(rng)
        L = oracle.OLayout(d)
        rank, off = _brute_map(d)
        ii, jj = np.meshgrid(np.arange(d.m), np.arange(d.n), indexing="ij")
        r, o = L.locate(ii.ravel(), jj.ravel())
        assert np.array_equal(r, rank.ravel()) and np.array_equal(o, off.ravel())
        # buffer size: one past the last element a rank stores
        for q in range(d.nranks):
            sel = rank.ravel() == q
            need = int(off.ravel()[sel].max()) + 1 if sel.any() else 0
            assert L.local_elems(q) == need


def test_descriptor_hand_example():
    """5 x 5 in 2 x 2 blocks on a 2 x 2 grid (row-major ranks), first block on
    process (1, 1), LLD 4.  Block rows 0, 1, 2 go to process rows 1, 0, 1, so
    process row 0 holds rows 2-3 and process row 1 rows 0-1 and 4; columns
    likewise.  Element (4, 0): process (1, 1) = rank 3, its local row 2 (third
    row it holds), local column 0: offset 2.  Element (0, 3): process (1, 0) =
    rank 2, local (0, 1): offset 0 + 1*4 = 4.  Element (2, 0): rank 1, offset 0.
    Buffer sizes: rank 0 holds 2 x 2 -> 1*4 + 2 = 6; rank 1 2 x 3 -> 10; rank 2
    3 x 2 -> 7; rank 3 3 x 3 -> 11."""
    d = synth.ScaLapack(5, 5, 2, 2, 1, 1, 4, 2, 2)
    L = oracle.OLayout(d)
    r, o = L.locate(np.array([4, 0, 2, 0]), np.array([0, 3, 0, 0]))
    assert list(r) == [3, 2, 1, 3] and list(o) == [2, 4, 0, 0]
    assert [L.local_elems(q) for q in range(4)] == [6, 10, 7, 11]


def test_zero_sources_and_tight_lld_equal_block_cyclic():
    """RSRC = CSRC = 0 with LLD equal to every process row's local rows is the
    plain block-cyclic layout (pinned elsewhere)."""
    for m, n, mb, nb, pr, pc, order in [(24, 18, 4, 3, 3, 2, "row"), (16, 40, 2, 5, 2, 4, "col")]:
        lld = m // pr
        d = synth.ScaLapack(m, n, mb, nb, 0, 0, lld, pr, pc, order)
        b = synth.BlockCyclic(m, n, mb, nb, pr, pc, order, "col")
        ii, jj = np.meshgrid(np.arange(m), np.arange(n), indexing="ij")
        x = oracle.OLayout(d).locate(ii.ravel(), jj.ravel())
        y = oracle.OLayout(b).locate(ii.ravel(), jj.ravel())
        assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])


def _gather(d, bufs):
    rank, off = _brute_map(d)
    g = np.zeros((d.m, d.n), bufs[0].dtype)
    for i, j in itertools.product(range(d.m), range(d.n)):
        g[i, j] = bufs[rank[i, j]][off[i, j]]
    return g


def _bufs(d, dtype, rng):
    L = oracle.OLayout(d)
    out = []
    for q in range(d.nranks):
        k = L.local_elems(q)
        v = rng.integers(-64, 64, size=k) / 8.0
        if dtype in ("c128", "c64"):
            v = v + 1j * (rng.integers(-64, 64, size=k) / 8.0)
        out.append(np.ascontiguousarray(v.astype(oracle.NUMPY[dtype])))
    return out


@pytest.mark.parametrize("routine", ["gemr2d", "tran", "tranc"])
@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
def test_scalapack_call_matches_global_slicing(routine, dtype):
    """sub(C) against numpy on the gathered global matrices; everything of C
    outside the window (other elements and the padding below each local
    matrix) is left as it was.  Scalars 2 - 1j and 0.5 keep every product
    exact, so the only rounding is the final sum, on both sides."""
    rng = np.random.default_rng({"gemr2d": 1, "tran": 2, "tranc": 3}[routine] * 10 + len(dtype))
    cplx = dtype in ("c128", "c64")
    for _ in range(12):
        P = int(rng.integers(1, 7))
        shapes = [(a, P // a) for a in range(1, P + 1) if P % a == 0]
        ga, gc = shapes[int(rng.integers(len(shapes)))], shapes[int(rng.integers(len(shapes)))]
        dA = _random_desc(rng, *ga)
        dC = _random_desc(rng, *gc)
        if routine == "gemr2d":
            m, n = min(dA.m, dC.m), min(dA.n, dC.n)
            ra, ca = m, n
        else:
            m, n = min(dA.n, dC.m), min(dA.m, dC.n)
            ra, ca = n, m
        m, n = int(rng.integers(0, m + 1)), int(rng.integers(0, n + 1))
        ra, ca = (m, n) if routine == "gemr2d" else (n, m)
        ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
        ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
        alpha, beta = (2 - 1j, 0.5) if cplx else (2.0, 0.5)
        call = synth.ScaLapackCall(routine, dtype, m, n, alpha, beta, dA, ia, ja, dC, ic, jc)
        A_bufs = _bufs(dA, dtype, rng)
        C_bufs = _bufs(dC, dtype, rng)
        C0 = [c.copy() for c in C_bufs]
        gA, gC0 = _gather(dA, A_bufs), _gather(dC, C_bufs)
        oracle.scalapack_call(call, A_bufs, C_bufs)
        want = gC0.copy()
        src = gA[ia - 1:ia - 1 + ra, ja - 1:ja - 1 + ca]
        win = (slice(ic - 1, ic - 1 + m), slice(jc - 1, jc - 1 + n))
        if routine == "gemr2d":
            want[win] = src
        else:
            op_src = src.T.conj() if routine == "tranc" else src.T
            want[win] = op_src * alpha + gC0[win] * beta
        assert np.array_equal(_gather(dC, C_bufs), want)
        # untouched storage: every buffer entry that is not a window element
        rank, off = _brute_map(dC)
        for q in range(dC.nranks):
            keep = np.ones(C_bufs[q].size, bool)
            sel = rank[win] == q
            keep[off[win][sel]] = False
            assert np.array_equal(C_bufs[q][keep], C0[q][keep])


def test_window_volume_matches_counting():
    rng = np.random.default_rng(35)
    for _ in range(20):
        dA = _random_desc(rng, 2, 2)
        dB = _random_desc(rng, 1, 4)
        op = "N" if rng.random() < 0.5 else "T"
        m = min(dA.m, dB.m if op == "N" else dB.n)
        n = min(dA.n, dB.n if op == "N" else dB.m)
        m, n = int(rng.integers(0, m + 1)), int(rng.integers(0, n + 1))
        ia, ja = int(rng.integers(0, dA.m - m + 1)), int(rng.integers(0, dA.n - n + 1))
        rb, cb = (m, n) if op == "N" else (n, m)
        ib, jb = int(rng.integers(0, dB.m - rb + 1)), int(rng.integers(0, dB.n - cb + 1))
        V = oracle.volume_window(oracle.OLayout(dA), ia, ja, oracle.OLayout(dB), ib, jb, m, n, op)
        ra, _ = _brute_map(dA)
        rbm, _ = _brute_map(dB)
        want = np.zeros((4, 4), np.int64)
        for i, j in itertools.product(range(m), range(n)):
            s = rbm[ib + i, jb + j] if op == "N" else rbm[ib + j, jb + i]
            want[s, ra[ia + i, ja + j]] += 1
        assert np.array_equal(V, want)


def _mapped(rng, d, world):
    """The descriptor on `world` ranks: its grid positions take distinct
    random ranks (column-major over the grid, like a BLACS user map)."""
    d.world = world
    d.rank_map = [int(x) for x in rng.permutation(world)[:d.nprow * d.npcol]]
    return d


def test_rank_map_storage_matches_dealing():
    """With a rank map the grid is any subset of a larger set of ranks; ranks
    outside it hold nothing."""
    rng = np.random.default_rng(36)
    for _ in range(40):
        d = _mapped(rng, _random_desc(rng), int(rng.integers(9, 14)))
        L = oracle.OLayout(d)
        rank, off = _brute_map(d)
        ii, jj = np.meshgrid(np.arange(d.m), np.arange(d.n), indexing="ij")
        r, o = L.locate(ii.ravel(), jj.ravel())
        assert np.array_equal(r, rank.ravel()) and np.array_equal(o, off.ravel())
        for q in range(d.world):
            sel = rank.ravel() == q
            assert L.local_elems(q) == (int(off.ravel()[sel].max()) + 1 if sel.any() else 0)
            if q not in d.rank_map:
                assert L.local_elems(q) == 0


def test_rank_map_identity_equals_rank_order():
    rng = np.random.default_rng(37)
    for order in ("row", "col"):
        d = _random_desc(rng, 2, 3, pad=1)
        d.rank_order = order
        e = synth.ScaLapack(d.m, d.n, d.mb, d.nb, d.rsrc, d.csrc, d.lld, 2, 3, "row", world=6,
                            rank_map=[(pr * 3 + pc) if order == "row" else (pr + pc * 2)
                                      for pc in range(3) for pr in range(2)])
        ii, jj = np.meshgrid(np.arange(d.m), np.arange(d.n), indexing="ij")
        x = oracle.OLayout(d).locate(ii.ravel(), jj.ravel())
        y = oracle.OLayout(e).locate(ii.ravel(), jj.ravel())
        assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])


@pytest.mark.parametrize("routine", ["gemr2d", "tran"])
def test_scalapack_call_between_grids_of_different_sizes(routine):
    """pxgemr2d / pxtran between a grid and a smaller (or one-process) grid of
    the same ranks, e.g. scattering a matrix held by one process."""
    rng = np.random.default_rng(38 if routine == "gemr2d" else 39)
    for trial in range(10):
        world = int(rng.integers(4, 9))
        shapes = [(1, 1), (1, 2), (2, 2), (2, 1), (1, 3), (3, 1), (2, 3)]
        ok = [g for g in shapes if g[0] * g[1] <= world]
        ga, gc = ok[int(rng.integers(len(ok)))], ok[int(rng.integers(len(ok)))]
        dA = _mapped(rng, _random_desc(rng, *ga), world)
        dC = _mapped(rng, _random_desc(rng, *gc), world)
        tr = routine != "gemr2d"
        m = min(dC.m, dA.n if tr else dA.m)
        n = min(dC.n, dA.m if tr else dA.n)
        m, n = int(rng.integers(0, m + 1)), int(rng.integers(0, n + 1))
        ra, ca = (n, m) if tr else (m, n)
        ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
        ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
        call = synth.ScaLapackCall(routine, "f64", m, n, 2.0, 0.5, dA, ia, ja, dC, ic, jc)
        A_bufs = _bufs(dA, "f64", rng)
        C_bufs = _bufs(dC, "f64", rng)
        gA, gC0 = _gather(dA, A_bufs), _gather(dC, C_bufs)
        oracle.scalapack_call(call, A_bufs, C_bufs)
        want = gC0.copy()
        src = gA[ia - 1:ia - 1 + ra, ja - 1:ja - 1 + ca]
        win = (slice(ic - 1, ic - 1 + m), slice(jc - 1, jc - 1 + n))
        want[win] = src if not tr else src.T * 2.0 + gC0[win] * 0.5
        assert np.array_equal(_gather(dC, C_bufs), want)
