"""GPU parity of the ScaLAPACK-compatible entry points (through the C ABI)
against the oracle's window transform: bit-exact over whole buffers (window
elements transformed, everything else untouched) at the reduced sizes and on
random descriptors, and at full size on every element of a few ranks plus
random points of all ranks."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2106_06601_amd as C

TORCH = {"f64": torch.float64, "c128": torch.complex128, "f32": torch.float32, "c64": torch.complex64}
UINT = {"f64": np.uint64, "c128": np.uint64, "f32": np.uint32, "c64": np.uint32}
ROUTINE_OP = {"gemr2d": "N", "tran": "T", "tranu": "T", "tranc": "C"}


def _say(msg):
    print(msg, flush=True)


def _bits(x, dtype):
    return np.ascontiguousarray(x).view(UINT[dtype])


def _grid(d):
    return (d.nprow, d.npcol, d.rank_order, d.world, d.rank_map)


class SLCase:
    """One ScaLAPACK-style call on the device.  Source buffers hold the
    generator's stream (B, 0, rank), destination buffers (A, 0, rank), both of
    the full descriptor's local size."""

    def __init__(self, call, seed=synth.DEFAULT_SEED, null_idle=False):
        self.call, self.seed = call, seed
        self.dev = torch.device("cuda:0")
        self.stream = torch.cuda.current_stream(self.dev)
        self.OA, self.OC = oracle.OLayout(call.A), oracle.OLayout(call.C)
        td = TORCH[call.dtype]
        self.a = [torch.empty(self.OA.local_elems(q), dtype=td, device=self.dev) for q in range(call.A.nranks)]
        self.c = [torch.empty(self.OC.local_elems(q), dtype=td, device=self.dev) for q in range(call.C.nranks)]
        h = self.stream.cuda_stream
        for q, t in enumerate(self.a):
            if t.numel():
                synth.fill_device(call.dtype, t.data_ptr(), t.numel(), seed, synth.stream(synth.ROLE_B, 0, q), h)
        for q, t in enumerate(self.c):
            if t.numel():
                synth.fill_device(call.dtype, t.data_ptr(), t.numel(), seed, synth.stream(synth.ROLE_A, 0, q), h)
        self.a_ptr, self.c_ptr = list(self.a), list(self.c)
        if null_idle:
            # ranks holding nothing of a submatrix may pass NULL
            tr = call.routine != "gemr2d"
            ra, ca = (call.n, call.m) if tr else (call.m, call.n)
            la = C.layout_from_spec(call.A).submatrix(call.ia - 1, call.ja - 1, ra, ca)
            lc = C.layout_from_spec(call.C).submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
            self.a_ptr = [t if la.local_elems(q) else None for q, t in enumerate(self.a)]
            self.c_ptr = [t if lc.local_elems(q) else None for q, t in enumerate(self.c)]

    def run(self, named=False):
        c = self.call
        ga, gc = _grid(c.A), _grid(c.C)
        s = self.stream
        if c.routine == "gemr2d":
            if named and c.dtype == "f64":
                C.costa_pdgemr2d(c.m, c.n, self.a_ptr, c.ia, c.ja, c.A.desc(), ga, self.c_ptr, c.ic, c.jc, c.C.desc(),
                                 gc, stream=s)
            else:
                C.costa_pxgemr2d(c.dtype, c.m, c.n, self.a_ptr, c.ia, c.ja, c.A.desc(), ga, self.c_ptr, c.ic, c.jc,
                                 c.C.desc(), gc, stream=s)
            return
        args = (c.m, c.n, c.alpha, self.a_ptr, c.ia, c.ja, c.A.desc(), ga, c.beta, self.c_ptr, c.ic, c.jc,
                c.C.desc(), gc)
        if named and c.dtype == "f64":
            C.costa_pdtran(*args, stream=s)
        elif named and c.dtype == "c128" and c.routine in ("tran", "tranu"):
            C.costa_pztranu(*args, stream=s)
        elif named and c.dtype == "c128":
            C.costa_pztranc(*args, stream=s)
        else:
            C.costa_pxtran(c.dtype, ROUTINE_OP[c.routine], *args, stream=s)

    def host_inputs(self):
        c, npt = self.call, oracle.NUMPY[self.call.dtype]
        ha, hc = [], []
        for q in range(c.A.nranks):
            x = np.zeros(self.OA.local_elems(q), npt)
            oracle.fill(c.dtype, x, self.seed, synth.stream(synth.ROLE_B, 0, q))
            ha.append(x)
        for q in range(c.C.nranks):
            x = np.zeros(self.OC.local_elems(q), npt)
            oracle.fill(c.dtype, x, self.seed, synth.stream(synth.ROLE_A, 0, q))
            hc.append(x)
        return ha, hc

    def check_full(self):
        torch.cuda.synchronize()
        ha, hc = self.host_inputs()
        oracle.scalapack_call(self.call, ha, hc)
        for q in range(self.call.C.nranks):
            got = self.c[q].cpu().numpy()
            bad = np.nonzero(_bits(got, self.call.dtype) != _bits(hc[q], self.call.dtype))[0]
            assert bad.size == 0, f"rank {q}: {bad.size} of {got.size} elements differ, first at {bad[:5]}"
        # the source is read only
        for q in range(self.call.A.nranks):
            assert np.array_equal(_bits(self.a[q].cpu().numpy(), self.call.dtype), _bits(ha[q], self.call.dtype))

    def check_ranks_and_samples(self, ranks, n_random=20000):
        """Every element of the given destination ranks (window elements from
        the oracle's expected values, the rest the untouched initial values),
        then random window points of all ranks."""
        torch.cuda.synchronize()
        c = self.call
        op = ROUTINE_OP[c.routine]
        alpha, beta = (1.0, 0.0) if c.routine == "gemr2d" else (c.alpha, c.beta)
        npt = oracle.NUMPY[c.dtype]
        wr = np.arange(c.m, dtype=np.int64)
        wc = np.arange(c.n, dtype=np.int64)
        # process row of each window row and process column of each window column
        rr, _ = self.OC.locate(wr + c.ic - 1, np.full(c.m, c.jc - 1))
        rc, _ = self.OC.locate(np.full(c.n, c.ic - 1), wc + c.jc - 1)
        if c.C.rank_map is not None:
            where = {rk: (k % c.C.nprow, k // c.C.nprow) for k, rk in enumerate(c.C.rank_map)}
            prow_of = np.vectorize(lambda r: where[int(r)][0])
            pcol_of = np.vectorize(lambda r: where[int(r)][1])
        elif c.C.rank_order == "row":
            prow_of, pcol_of = (lambda r: r // c.C.npcol), (lambda r: r % c.C.npcol)
        else:
            prow_of, pcol_of = (lambda r: r % c.C.nprow), (lambda r: r // c.C.nprow)
        for q in ranks:
            pr, pc = prow_of(q), pcol_of(q)
            rows = wr[prow_of(rr) == pr]
            cols = wc[pcol_of(rc) == pc]
            ii, jj = np.meshgrid(rows, cols, indexing="ij")
            rank, off, val = oracle.expect_at_window(c.dtype, op, alpha, beta, self.OC, c.ic - 1, c.jc - 1,
                                                     self.OA, c.ia - 1, c.ja - 1, self.seed, 0, ii.ravel(),
                                                     jj.ravel())
            assert np.all(rank == q)
            want = np.zeros(self.OC.local_elems(q), npt)
            oracle.fill(c.dtype, want, self.seed, synth.stream(synth.ROLE_A, 0, q))
            want[off] = val
            got = self.c[q].cpu().numpy()
            bad = np.nonzero(_bits(got, c.dtype) != _bits(want, c.dtype))[0]
            assert bad.size == 0, f"rank {q}: {bad.size} of {got.size} elements differ, first at {bad[:5]}"
        rng = np.random.default_rng(5)
        ri, rj = rng.integers(0, c.m, n_random), rng.integers(0, c.n, n_random)
        ri[:4], rj[:4] = [0, c.m - 1, 0, c.m - 1], [0, 0, c.n - 1, c.n - 1]
        rank, off, val = oracle.expect_at_window(c.dtype, op, alpha, beta, self.OC, c.ic - 1, c.jc - 1, self.OA,
                                                 c.ia - 1, c.ja - 1, self.seed, 0, ri, rj)
        for q in np.unique(rank):
            sel = rank == q
            got = self.c[q][torch.from_numpy(off[sel]).to(self.dev)].cpu().numpy()
            assert np.array_equal(_bits(got, c.dtype), _bits(val[sel], c.dtype)), f"rank {q} samples differ"


@pytest.mark.parametrize("name", synth.SCALAPACK_CALLS)
def test_scalapack_small_matches_oracle(name):
    call = synth.scalapack_call(name, "small")
    _say(f"scalapack {name} small")
    k = SLCase(call)
    k.run(named=True)
    k.check_full()


def _random_call(seed):
    rng = np.random.default_rng(1000 + seed)
    routine = ["gemr2d", "tran", "tranu", "tranc"][seed % 4]
    dtype = ["f64", "c128", "f32", "c64"][(seed // 4) % 4]
    P = [4, 6, 8, 12][seed % 4]
    shapes = [(a, P // a) for a in range(1, P + 1) if P % a == 0]

    def desc(grid):
        m, n = int(rng.integers(1, 400)), int(rng.integers(1, 400))
        mb, nb = int(rng.integers(1, 70)), int(rng.integers(1, 70))
        rsrc, csrc = int(rng.integers(0, grid[0])), int(rng.integers(0, grid[1]))
        lr = max(oracle.numroc(m, mb, p, rsrc, grid[0]) for p in range(grid[0]))
        return synth.ScaLapack(m, n, mb, nb, rsrc, csrc, max(1, lr) + int(rng.integers(0, 5)), grid[0], grid[1],
                               "row" if rng.random() < 0.5 else "col")

    dA = desc(shapes[int(rng.integers(len(shapes)))])
    dC = desc(shapes[int(rng.integers(len(shapes)))])
    tr = routine != "gemr2d"
    mmax, nmax = min(dC.m, dA.n if tr else dA.m), min(dC.n, dA.m if tr else dA.n)
    m, n = int(rng.integers(1, mmax + 1)), int(rng.integers(1, nmax + 1))
    ra, ca = (n, m) if tr else (m, n)
    ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
    ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
    cplx = dtype in ("c128", "c64")
    alpha, beta = [(2 - 1j, 0.5), (1.0, 0.0), (0.5j, 1.0), (-1.0, 0.0)][seed % 4] if cplx else \
        [(2.0, 0.5), (1.0, 0.0), (-0.5, 1.0), (3.0, 0.0)][seed % 4]
    return synth.ScaLapackCall(routine, dtype, m, n, alpha, beta, dA, ia, ja, dC, ic, jc)


@pytest.mark.parametrize("seed", range(16))
def test_scalapack_random_calls(seed):
    call = _random_call(seed)
    _say(f"scalapack random {seed}: {call.routine} {call.dtype} {call.m}x{call.n}")
    k = SLCase(call, seed=seed, null_idle=seed % 2 == 1)
    k.run()
    k.check_full()


@pytest.mark.parametrize("name", synth.SCALAPACK_CALLS)
def test_scalapack_full_size(name):
    call = synth.scalapack_call(name)
    _say(f"scalapack {name} full")
    k = SLCase(call)
    k.run(named=True)
    if call.beta == 0:
        k.run(named=True)  # the cached plan again: the same result
    P = call.C.nranks
    held = [q for q in range(P) if k.OC.local_elems(q)]
    k.check_ranks_and_samples(sorted({held[0], held[1 % len(held)], held[len(held) // 2], held[-1]}))


def test_scalapack_alternating_windows_and_empty_calls():
    """Two windows of the same descriptors in turn, through the cached layouts
    and plans; empty calls enqueue nothing."""
    base = synth.scalapack_call("pdtran_16k", "small")
    _say("scalapack alternating windows")
    calls = [base,
             synth.ScaLapackCall("tran", "f64", 700, 900, 2.0, 0.5, base.A, 301, 5, base.C, 129, 1000),
             base]
    for i, call in enumerate(calls):
        k = SLCase(call, seed=77 + i)
        k.run(named=True)
        k.check_full()
    k = SLCase(base, seed=80)
    C.costa_pdtran(0, 5, 1.0, k.a, 1, 1, base.A.desc(), _grid(base.A), 0.0, k.c, 1, 1, base.C.desc(),
                   _grid(base.C), stream=k.stream)
    C.costa_pdgemr2d(5, 0, k.a, 1, 1, base.A.desc(), _grid(base.A), k.c, 1, 1, base.C.desc(), _grid(base.C),
                     stream=k.stream)
    torch.cuda.synchronize()
    _, hc = k.host_inputs()
    for q in range(base.C.nranks):
        assert np.array_equal(_bits(k.c[q].cpu().numpy(), "f64"), _bits(hc[q], "f64"))


@pytest.mark.parametrize("seed", range(6))
def test_window_volume_matrix_matches_oracle(seed):
    """costa_volume_matrix on submatrix layouts: the separable path (both
    block-cyclic) and the overlay kernel (a general grid's window)."""
    rng = np.random.default_rng(2000 + seed)
    call = _random_call(seed)
    op = ROUTINE_OP[call.routine]
    ra, ca = (call.n, call.m) if op != "N" else (call.m, call.n)
    LA = C.layout_from_spec(call.A).submatrix(call.ia - 1, call.ja - 1, ra, ca)
    LC = C.layout_from_spec(call.C).submatrix(call.ic - 1, call.jc - 1, call.m, call.n)
    _say(f"window volume {seed}")
    V = C.costa_volume_matrix(LC, LA, op)
    want = oracle.volume_window(oracle.OLayout(call.C), call.ic - 1, call.jc - 1, oracle.OLayout(call.A),
                                call.ia - 1, call.ja - 1, call.m, call.n, op)
    assert np.array_equal(V, want)
    # a general grid's window as the source
    P = call.C.nranks
    M, N = ra + int(rng.integers(0, 50)), ca + int(rng.integers(0, 50))
    rs = [0] + sorted(rng.choice(np.arange(1, M), min(M - 1, 7), replace=False).tolist()) + [M]
    cs = [0] + sorted(rng.choice(np.arange(1, N), min(N - 1, 5), replace=False).tolist()) + [N]
    G = synth.General(M, N, rs, cs, rng.integers(0, P, (len(rs) - 1) * (len(cs) - 1)).tolist(), P, "row")
    i0, j0 = int(rng.integers(0, M - ra + 1)), int(rng.integers(0, N - ca + 1))
    LG = C.layout_from_spec(G).submatrix(i0, j0, ra, ca)
    V = C.costa_volume_matrix(LC, LG, op)
    want = oracle.volume_window(oracle.OLayout(call.C), call.ic - 1, call.jc - 1, oracle.OLayout(G), i0, j0,
                                call.m, call.n, op)
    assert np.array_equal(V, want)


@pytest.mark.parametrize("seed", range(8))
def test_scalapack_between_grids_of_different_sizes(seed):
    """pxgemr2d / pxtran between grids of different shapes over one set of
    ranks (BLACS-style rank maps): scatter from one process, gather to one
    process, mixed grids; ranks outside a grid pass NULL."""
    rng = np.random.default_rng(4000 + seed)
    routine = ["gemr2d", "tran", "tranc", "gemr2d"][seed % 4]
    dtype = ["f64", "c128"][(seed // 4) % 2]
    world = int(rng.integers(6, 17))
    pairs = [((1, 1), (2, 3)), ((2, 3), (1, 1)), ((1, 2), (3, 2)), ((2, 2), (1, 3))]
    ga, gc = pairs[seed % len(pairs)]

    def desc(grid):
        m, n = int(rng.integers(1, 300)), int(rng.integers(1, 300))
        mb, nb = int(rng.integers(1, 50)), int(rng.integers(1, 50))
        rsrc, csrc = int(rng.integers(0, grid[0])), int(rng.integers(0, grid[1]))
        lr = max(oracle.numroc(m, mb, p, rsrc, grid[0]) for p in range(grid[0]))
        return synth.ScaLapack(m, n, mb, nb, rsrc, csrc, max(1, lr) + 3, grid[0], grid[1], "row", world=world,
                               rank_map=[int(x) for x in rng.permutation(world)[:grid[0] * grid[1]]])

    dA, dC = desc(ga), desc(gc)
    tr = routine != "gemr2d"
    mmax, nmax = min(dC.m, dA.n if tr else dA.m), min(dC.n, dA.m if tr else dA.n)
    m, n = int(rng.integers(1, mmax + 1)), int(rng.integers(1, nmax + 1))
    ra, ca = (n, m) if tr else (m, n)
    ia, ja = int(rng.integers(1, dA.m - ra + 2)), int(rng.integers(1, dA.n - ca + 2))
    ic, jc = int(rng.integers(1, dC.m - m + 2)), int(rng.integers(1, dC.n - n + 2))
    alpha, beta = (2 - 1j, 0.5) if dtype == "c128" else (2.0, 0.5)
    call = synth.ScaLapackCall(routine, dtype, m, n, alpha, beta, dA, ia, ja, dC, ic, jc)
    _say(f"scalapack grids {ga} -> {gc} of {world} ranks: {routine} {dtype} {m}x{n}")
    k = SLCase(call, seed=seed, null_idle=True)
    k.run()
    k.check_full()
    # the volume matrix of the two rank-mapped windows (separable kernels,
    # ranks outside a grid send or receive nothing) against brute-force counting
    op = ROUTINE_OP[routine]
    LA = C.layout_from_spec(dA).submatrix(ia - 1, ja - 1, ra, ca)
    LC = C.layout_from_spec(dC).submatrix(ic - 1, jc - 1, m, n)
    V = C.costa_volume_matrix(LC, LA, op)
    want = oracle.volume_window(oracle.OLayout(dC), ic - 1, jc - 1, oracle.OLayout(dA), ia - 1, ja - 1, m, n, op)
    assert np.array_equal(V, want)


def test_many_windows_pass_the_layout_cache_bound():
    """1156 calls on distinct 8 x 8 windows of two 48 x 48 matrices, about
    2300 distinct window layouts -- more than the library keeps, so its
    layout cache starts over during the sequence: the final buffers equal
    the same window copies applied in order on the host (through the
    oracle's storage maps), and nothing outside the windows is touched."""
    import itertools
    SL = synth.ScaLapack
    A = SL(48, 48, 5, 7, 0, 1, 27, 2, 2)   # local rows 25 / 23, lld padded to 27
    Cd = SL(48, 48, 4, 6, 1, 0, 24, 2, 2, rank_order="col")
    OA, OC = oracle.OLayout(A), oracle.OLayout(Cd)
    dev = torch.device("cuda:0")
    s = torch.cuda.current_stream(dev)
    ha, hc = [], []
    for q in range(4):
        a = np.zeros(OA.local_elems(q))
        oracle.fill("f64", a, 5, synth.stream(synth.ROLE_B, 0, q))
        ha.append(a)
        c = np.zeros(OC.local_elems(q))
        oracle.fill("f64", c, 5, synth.stream(synth.ROLE_A, 0, q))
        hc.append(c)
    da = [torch.from_numpy(a).to(dev) for a in ha]
    dc = [torch.from_numpy(c).to(dev) for c in hc]
    ii, jj = np.meshgrid(np.arange(8), np.arange(8), indexing="ij")
    ii, jj = ii.ravel(), jj.ravel()
    _say("ScaLAPACK-style calls on 1156 distinct windows")
    for i0, j0 in itertools.product(range(34), range(34)):
        ic0, jc0 = (i0 * 7) % 41, (j0 * 5) % 41
        C.costa_pxgemr2d("f64", 8, 8, da, i0 + 1, j0 + 1, A.desc(), _grid(A), dc, ic0 + 1, jc0 + 1, Cd.desc(),
                         _grid(Cd), stream=s)
        ra, oa = OA.locate(ii + i0, jj + j0)
        rc, oc = OC.locate(ii + ic0, jj + jc0)
        for k in range(ii.size):
            hc[rc[k]][oc[k]] = ha[ra[k]][oa[k]]
    torch.cuda.synchronize()
    for q in range(4):
        assert np.array_equal(_bits(dc[q].cpu().numpy(), "f64"), _bits(hc[q], "f64")), f"rank {q}"
