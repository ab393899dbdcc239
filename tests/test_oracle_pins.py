"""Pins of the CPU oracle against what the paper and plain mathematics fix.

None of these compares the oracle with itself: each check uses a closed form,
an invariant proved in the paper, a textbook routine (numpy dense ops, scipy's
assignment solver), brute force, or a value the paper prints.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
BC = synth.BlockCyclic
GEN = synth.General


# ---------------------------------------------------------------------------
# the input generator
# ---------------------------------------------------------------------------
def test_generator_copies_agree_and_grid():
    strm = synth.stream(synth.ROLE_B, 3, 17)
    a = synth.values("f64", 99, strm, 4096)
    b = np.zeros(4096)
    oracle.fill("f64", b, 99, strm)
    assert np.array_equal(a.view(np.uint64), b.view(np.uint64))
    # scalar definition for a few entries
    for k in (0, 1, 4095):
        bits = synth.bits(99, strm, k)
        assert a[k] == 2.0 * ((bits >> 11) * 2.0**-53) - 1.0
    assert a.min() >= -1.0 and a.max() < 1.0
    assert not np.any(np.signbit(a) & (a == 0))  # never -0
    assert np.all((a * 2.0**52) == np.round(a * 2.0**52))  # on the 2^-52 grid
    c = synth.values("c128", 99, strm, 64)
    cc = np.zeros(64, dtype=np.complex128)
    oracle.fill("c128", cc, 99, strm)
    assert np.array_equal(c, cc)


def test_random_cuts_distinct_sorted_in_range():
    cuts = synth.random_cuts(5, 77, 16384, 40)
    assert len(cuts) == 40 and len(set(cuts)) == 40
    assert cuts == sorted(cuts) and cuts[0] >= 1 and cuts[-1] <= 16383
    assert synth.random_cuts(5, 77, 41, 40) == list(range(1, 41))  # every interior point


# ---------------------------------------------------------------------------
# storage maps (Section 5 layout; Section 6 Figure 1 local view)
# ---------------------------------------------------------------------------
def _all_points(spec):
    ii, jj = np.meshgrid(np.arange(spec.nrows), np.arange(spec.ncols), indexing="ij")
    return ii.ravel(), jj.ravel()


LAYOUTS = [
    BC(37, 53, 4, 8, 3, 2, "row", "col"),
    BC(37, 53, 4, 8, 3, 2, "col", "row"),
    BC(64, 64, 16, 16, 2, 2, "row", "col"),
    BC(10, 7, 3, 2, 4, 3, "row", "col"),   # some ranks hold nothing in one dimension
    GEN(11, 9, [0, 3, 4, 11], [0, 5, 9], [2, 0, 1, 1, 2, 0], 3, "col"),
    GEN(11, 9, [0, 3, 4, 11], [0, 5, 9], [2, 0, 1, 1, 2, 0], 3, "row"),
]


@pytest.mark.parametrize("spec", LAYOUTS, ids=lambda s: f"{s.kind}-{s.block_order}")
def test_storage_map_is_a_bijection(spec):
    L = oracle.OLayout(spec)
    i, j = _all_points(spec)
    rank, off = L.locate(i, j)
    sizes = [L.local_elems(r) for r in range(spec.nranks)]
    assert sum(sizes) == spec.nrows * spec.ncols
    assert np.all(off >= 0)
    assert np.all(off < np.asarray(sizes)[rank])
    keys = rank.astype(np.int64) * (1 << 40) + off
    assert np.unique(keys).size == keys.size  # every element has its own slot


def test_numroc_exact_counts():
    L = oracle.OLayout(BC(20000, 20000, 64, 64, 8, 4, "row", "col"))
    # rank = pr*4 + pc
    assert L.local_elems(0) == 2528 * 5024          # pr 0, pc 0
    assert L.local_elems(1) == 2528 * 4992          # pr 0, pc 1
    assert L.local_elems(4) == 2496 * 5024          # pr 1, pc 0
    assert L.local_elems(31) == 2496 * 4992         # pr 7, pc 3
    T = oracle.OLayout(BC(20000, 20000, 100, 100, 4, 8, "row", "row"))
    assert all(T.local_elems(r) == 5000 * 2500 for r in range(32))


def test_hand_computed_addresses():
    # 1024^2, 32x32 blocks on a 2x2 grid, row-major ranks, col-major storage.
    # (40, 70): block row 1 -> pr 1, block col 2 -> pc 0, rank 2;
    # local row 8, local col 32 + 6 = 38, 512 local rows -> offset 8 + 38*512.
    L = oracle.OLayout(BC(1024, 1024, 32, 32, 2, 2, "row", "col"))
    r, o = L.locate(np.array([40]), np.array([70]))
    assert (r[0], o[0]) == (2, 8 + 38 * 512)
    # 64x64 blocks, col-major ranks: (40, 70) is in block (0, 1): pr 0, pc 1,
    # rank 0 + 1*2 = 2; local (40, 6), offset 40 + 6*512.
    L2 = oracle.OLayout(BC(1024, 1024, 64, 64, 2, 2, "col", "col"))
    r, o = L2.locate(np.array([40]), np.array([70]))
    assert (r[0], o[0]) == (2, 40 + 6 * 512)
    # row-major storage of 100x100 blocks on 4x8 (row-major ranks), 2500 local cols:
    # (250, 1234): pr (2)%4 = 2, pc 12%8 = 4 -> rank 20; local (50, 1*100+34=134)
    L3 = oracle.OLayout(BC(20000, 20000, 100, 100, 4, 8, "row", "row"))
    r, o = L3.locate(np.array([250]), np.array([1234]))
    assert (r[0], o[0]) == (20, 50 * 2500 + 134)
    # general grid: rows [0,3,4,11], cols [0,5,9], owners row-major [[2,0],[1,1],[2,0]];
    # rank 2 stores block (0,0) (3x5) then block (2,0) (7x5); col-major, ld = block rows.
    G = oracle.OLayout(GEN(11, 9, [0, 3, 4, 11], [0, 5, 9], [2, 0, 1, 1, 2, 0], 3, "col"))
    r, o = G.locate(np.array([5, 1]), np.array([2, 4]))
    assert (r[0], o[0]) == (2, 15 + (5 - 4) + 2 * 7)
    assert (r[1], o[1]) == (2, 1 + 4 * 3)


# ---------------------------------------------------------------------------
# volume matrix (Section 2 volumes, Algorithm 2 packages)
# ---------------------------------------------------------------------------
def _separable_volume(A, B, op):
    """The oracle's per-dimension count (pinned below against the
    element-by-element count and closed forms)."""
    return oracle.volume_separable(A, B, op)


def _check_conservation(V, A, B, op):
    LA, LB = oracle.OLayout(A), oracle.OLayout(B)
    P = V.shape[0]
    assert V.sum() == A.nrows * A.ncols
    assert all(V[s].sum() == LB.local_elems(s) for s in range(P))
    assert all(V[:, t].sum() == LA.local_elems(t) for t in range(P))


def test_volume_reshuffle_transpose_1k_closed_form():
    w = synth.workload("reshuffle_transpose_1k")
    it = w.items[0]
    V = oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op)
    assert np.all(V == 65536)  # every 64-block of A takes 16 32-blocks, 4 from each rank
    _check_conservation(V, it.A, it.B, it.op)
    assert np.array_equal(V, _separable_volume(it.A, it.B, it.op))


def test_volume_blocksize_change_closed_form():
    w = synth.workload("blocksize_change_16k", "small")
    it = w.items[0]
    V = oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op)
    n = it.A.nrows
    unit = n * n // 64
    for s in range(16):
        for t in range(16):
            sr, sc, tr, tc = s // 4, s % 4, t // 4, t % 4
            ok = sr in (2 * (tr % 2), 2 * (tr % 2) + 1) and sc in (2 * (tc % 2), 2 * (tc % 2) + 1)
            assert V[s, t] == (unit if ok else 0)
    _check_conservation(V, it.A, it.B, it.op)


@pytest.mark.parametrize("k", [0, 4])
def test_volume_rpa_items_closed_form(k):
    w = synth.workload("rpa_batched_tall_skinny", "small")
    it = w.items[k]
    V = oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op)
    assert np.array_equal(V, _separable_volume(it.A, it.B, it.op))
    unit = 512 * 64
    for s in range(64):
        for t in range(64):
            hit = (s // 8 == t % 8) if it.op == "N" else (s // 8 == t // 8)
            assert V[s, t] == (unit if hit else 0)
    _check_conservation(V, it.A, it.B, it.op)


def test_volume_scaled_transpose_matches_separable_small():
    w = synth.workload("scaled_transpose_20k", "small")
    it = w.items[0]
    V = oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op)
    assert np.array_equal(V, _separable_volume(it.A, it.B, it.op))
    _check_conservation(V, it.A, it.B, it.op)


def test_volume_separable_matches_bruteforce_rectangular_blocks():
    """The per-dimension count against element-by-element counting on
    block-cyclic layouts with non-square blocks, both rank orders and all
    ops (a transposed op reads B's column blocks along A's rows)."""
    rng = np.random.default_rng(6)
    for case in range(12):
        op = "NTC"[case % 3]
        M, N = int(rng.integers(20, 60)), int(rng.integers(20, 60))
        pa = [(1, 6), (2, 3), (3, 2), (6, 1)][int(rng.integers(0, 4))]
        pb = [(1, 6), (2, 3), (3, 2), (6, 1)][int(rng.integers(0, 4))]
        a, b = int(rng.integers(1, 7)), int(rng.integers(1, 7))
        A = BC(M, N, a, a + int(rng.integers(1, 4)), pa[0], pa[1], ["row", "col"][case % 2], "col")
        bm, bn = (M, N) if op == "N" else (N, M)
        B = BC(bm, bn, b + int(rng.integers(1, 4)), b, pb[0], pb[1], ["col", "row"][(case // 2) % 2], "row")
        V = oracle.volume(oracle.OLayout(A), oracle.OLayout(B), op)
        assert np.array_equal(V, _separable_volume(A, B, op)), (case, A, B, op)
        _check_conservation(V, A, B, op)


def test_volume_scaled_transpose_full_size_retained():
    # full 20000^2 by per-dimension counting: identity keeps 12,500,384 elements
    # local, the optimal relabeling 13,407,488
    w = synth.workload("scaled_transpose_20k")
    it = w.items[0]
    V = _separable_volume(it.A, it.B, it.op)
    assert V.sum() == 20000 * 20000
    assert np.trace(V) == 12500384
    assert oracle.retained(V, oracle.relabel_exact(V)) == 13407488


def test_volume_general_grid_bruteforce_tiny():
    A = GEN(7, 6, [0, 2, 7], [0, 1, 6], [0, 1, 1, 0], 2, "col")
    B = GEN(6, 7, [0, 3, 6], [0, 4, 7], [1, 1, 0, 1], 2, "row")
    V = oracle.volume(oracle.OLayout(A), oracle.OLayout(B), "T")
    # count by hand from the definitions: A(i,j) reads B(j,i)
    ownA = lambda i, j: [[0, 1], [1, 0]][0 if i < 2 else 1][0 if j < 1 else 1]
    ownB = lambda i, j: [[1, 1], [0, 1]][0 if i < 3 else 1][0 if j < 4 else 1]
    ref = np.zeros((2, 2), np.int64)
    for i in range(7):
        for j in range(6):
            ref[ownB(j, i), ownA(i, j)] += 1
    assert np.array_equal(V, ref)


# ---------------------------------------------------------------------------
# relabeling (Section 4)
# ---------------------------------------------------------------------------
def _rand_V(rng, P, zero_frac=0.3, hi=50):
    V = rng.integers(0, hi, size=(P, P)).astype(np.int64)
    V[rng.random((P, P)) < zero_frac] = 0
    return V


def test_relabel_bruteforce_dp_scipy_agree():
    rng = np.random.default_rng(1)
    for P in range(1, 8):
        for _ in range(4):
            V = _rand_V(rng, P, hi=4)  # small range -> many ties
            s1 = oracle.relabel_bruteforce(V)
            assert oracle.relabel_dp(V) == s1
            assert oracle.relabel_exact(V) == s1
    for P in (10, 13):
        V = _rand_V(rng, P, hi=5)
        assert oracle.relabel_dp(V) == oracle.relabel_exact(V)


def test_relabel_optimum_value_matches_scipy_and_beats_identity():
    from scipy.optimize import linear_sum_assignment
    rng = np.random.default_rng(2)
    for P in (5, 9, 16):
        V = _rand_V(rng, P, hi=1000)
        sig = oracle.relabel(V)
        assert sorted(sig) == list(range(P))
        r, c = linear_sum_assignment(V, maximize=True)
        assert oracle.retained(V, sig) == int(V[r, c].sum())
        # the identity is always a perfect matching (Remark after Theorem 2)
        assert oracle.retained(V, sig) >= oracle.retained(V, list(range(P)))


def test_relabel_tie_break_is_lexicographic_min():
    V = np.full((4, 4), 7, np.int64)  # every relabeling is optimal
    assert oracle.relabel(V) == [0, 1, 2, 3]
    V = np.array([[0, 5], [5, 0]], np.int64)
    assert oracle.relabel(V) == [1, 0]


def test_lemma1_total_gain_equals_cost_difference():
    rng = np.random.default_rng(3)
    for P in (3, 6, 9):
        V = _rand_V(rng, P)
        ident = list(range(P))
        for _ in range(5):
            sig = list(rng.permutation(P))
            assert oracle.total_gain(V, sig) == oracle.total_cost(V, ident) - oracle.total_cost(V, sig)


def test_remark_gain_closed_form():
    rng = np.random.default_rng(4)
    V = _rand_V(rng, 7)
    for x in range(7):
        for y in range(7):
            assert oracle.gain(V, x, y) == int(V[y, x]) - int(V[x, x])


def test_topology_cost_hand_example():
    """P = 2 under the latency-bandwidth cost of Section 3: rank 0 sends 5
    elements to label 1, rank 1 sends 3 to label 0, latency 2 and 1 unit per
    byte between the two ranks, nothing within a rank.  By hand: identity
    W = (2 + 5) + (2 + 3) = 12; swapping the labels makes both packages
    local, W = 0; delta(p_0, p_1) = w(1,0,3) - w(1,1,3) = 5 and
    delta(p_1, p_0) = w(0,1,5) - w(0,0,5) = 7 (eq:delta)."""
    V = np.array([[0, 5], [3, 0]], np.int64)
    w = oracle.w_topology(np.array([[0.0, 2.0], [2.0, 0.0]]), np.array([[0.0, 1.0], [1.0, 0.0]]), 1.0)
    assert oracle.total_cost(V, [0, 1], w) == 12 and oracle.total_cost(V, [1, 0], w) == 0
    assert oracle.gain(V, 0, 1, w) == 5 and oracle.gain(V, 1, 0, w) == 7
    assert oracle.relabel_bruteforce_cost(V, w) == [1, 0]
    assert oracle.relabel_greedy(V, w) == [1, 0]
    # asymmetric links: only the bandwidth term of the used direction counts
    w2 = oracle.w_topology(np.zeros((2, 2)), np.array([[0.0, 1.0], [10.0, 0.0]]), 2.0)
    assert oracle.total_cost(V, [0, 1], w2) == 5 * 2 * 1.0 + 3 * 2 * 10.0


def test_greedy_hand_example_is_suboptimal():
    """Locally-free cost, P = 3, by hand: label 0 receives 5 from rank 1 and
    4 from rank 2; label 2 receives 4 from rank 1.  The gains are
    delta(p_x, p_y) = V[y][x] - V[x][x]: the heaviest edge (0 -> 1, gain 5)
    is taken first and blocks both edges of gain 4, so the greedy matching
    keeps 5 elements local (sigma = [1, 0, 2], W = 13 - 5 = 8) while the
    optimum keeps 8 (sigma = [2, 0, 1], W = 5) -- within the factor 2 of a
    greedy matching."""
    V = np.array([[0, 0, 0], [5, 0, 4], [4, 0, 0]], np.int64)
    assert oracle.total_cost(V, [0, 1, 2]) == 13
    g = oracle.relabel_greedy(V)
    assert g == [1, 0, 2]
    assert oracle.retained(V, g) == 5 and oracle.total_cost(V, g) == 8
    opt = oracle.relabel_bruteforce(V)
    assert opt == [2, 0, 1]
    assert oracle.retained(V, opt) == 8 and oracle.total_cost(V, opt) == 5


def test_greedy_keeps_the_identity_when_its_matching_loses():
    """Locally-free cost, P = 2, by hand: V = [[7, 2], [0, 0]].  Gains
    delta(p_x, p_y) = V[y][x] - V[x][x]: delta(p_1, p_0) = 2 is the only
    positive edge; taking it leaves (p_0, p_1) with delta = 0 - 7 = -7, a
    perfect matching of total gain -5 that moves 7 local elements off their
    rank to keep 2.  The identity (gain 0) is the result."""
    V = np.array([[7, 2], [0, 0]], np.int64)
    assert oracle.gain(V, 1, 0) == 2 and oracle.gain(V, 0, 1) == -7
    assert oracle.total_gain(V, [1, 0]) == -5
    assert oracle.relabel_greedy(V) == [0, 1]
    assert oracle.relabel_bruteforce(V) == [0, 1]


def test_greedy_is_a_two_approximation_and_never_loses():
    """A greedy matching on non-negative weights has at least half the
    weight of a maximum matching (the bound Section 6 relies on): checked
    against brute force over all P! relabelings wherever every gain is >= 0
    (volume matrices with an empty diagonal under the locally-free cost).
    For any volumes and either cost the result is never worse than the
    identity (Lemma 1: total gain = W(G) - W(G_sigma))."""
    rng = np.random.default_rng(5)
    for P in range(2, 7):
        for _ in range(6):
            V = _rand_V(rng, P, hi=9)
            ident = list(range(P))
            g = oracle.relabel_greedy(V)
            assert sorted(g) == ident
            assert oracle.total_gain(V, g) >= 0
            assert oracle.total_cost(V, g) <= oracle.total_cost(V, ident)
            Z = V.copy()
            np.fill_diagonal(Z, 0)
            assert all(oracle.gain(Z, x, y) >= 0 for x in range(P) for y in range(P))
            best = max(oracle.total_gain(Z, list(p)) for p in itertools.permutations(range(P)))
            assert 2 * oracle.total_gain(Z, oracle.relabel_greedy(Z)) >= best
            L = rng.random((P, P)) * 3
            Bw = rng.random((P, P))
            np.fill_diagonal(L, 0.0)
            np.fill_diagonal(Bw, 0.0)
            w = oracle.w_topology(L, Bw, 8.0)
            sg = oracle.relabel_greedy(V, w)
            assert sorted(sg) == ident
            assert oracle.total_cost(V, sg, w) <= oracle.total_cost(V, ident, w) + 1e-9


def test_blocksize_change_canonical_relabeling():
    # full-size volume pattern (closed form, 4,194,304 per non-zero pair); the
    # optimum keeps 25% local, identity 6.25%
    unit = 16384 * 16384 // 64
    V = np.zeros((16, 16), np.int64)
    for s in range(16):
        for t in range(16):
            sr, sc, tr, tc = s // 4, s % 4, t // 4, t % 4
            if sr in (2 * (tr % 2), 2 * (tr % 2) + 1) and sc in (2 * (tc % 2), 2 * (tc % 2) + 1):
                V[s, t] = unit
    sig = oracle.relabel(V)
    assert sig == [0, 2, 1, 3, 8, 10, 9, 11, 4, 6, 5, 7, 12, 14, 13, 15]
    assert oracle.retained(V, list(range(16))) == 16777216
    assert oracle.retained(V, sig) == 67108864


def test_paper_bench2_equal_blocks_full_relabeling():
    g = json.load(open(os.path.join(GOLDEN, "bench2_equal_blocks.json")))
    n, bs, p = g["matrix"][0], g["source"]["block"], g["grid"][0]
    A = BC(n, n, bs, bs, p, p, g["target"]["rank_order"], "col")
    B = BC(n, n, bs, bs, p, p, g["source"]["rank_order"], "col")
    V = _separable_volume(A, B, "N")
    sig = oracle.relabel(V)
    before = V.sum() - oracle.retained(V, list(range(p * p)))
    after = V.sum() - oracle.retained(V, sig)
    assert before == 9 * 10**9
    assert 100 * (before - after) // before == g["volume_reduction_percent"]
    # the same at a size the element-by-element count handles
    A2 = BC(1000, 1000, 100, 100, 10, 10, "col", "col")
    B2 = BC(1000, 1000, 100, 100, 10, 10, "row", "col")
    V2 = oracle.volume(oracle.OLayout(A2), oracle.OLayout(B2), "N")
    assert V2.sum() - oracle.retained(V2, oracle.relabel(V2)) == 0


# ---------------------------------------------------------------------------
# the transform, equation (eq:costa)
# ---------------------------------------------------------------------------
def _bufs(spec, dtype, role, seed=11, fill=True):
    L = oracle.OLayout(spec)
    out = []
    for r in range(spec.nranks):
        a = np.zeros(L.local_elems(r), dtype=oracle.NUMPY[dtype])
        if fill:
            oracle.fill(dtype, a, seed, synth.stream(role, 0, r))
        out.append(a)
    return L, out


def _dense_from_single_block(buf, spec):
    if spec.block_order == "col":
        return buf.reshape(spec.ncols, spec.nrows).T
    return buf.reshape(spec.nrows, spec.ncols)


@pytest.mark.parametrize("dtype", ["f64", "c128", "f32", "c64"])
@pytest.mark.parametrize("op", ["N", "T", "C"])
@pytest.mark.parametrize("orders", [("col", "col"), ("row", "col"), ("col", "row")])
@pytest.mark.parametrize("ab", [(1.0, 0.0), (-2.0, 0.0), (2.0, 0.5), (-0.5, 0.25), ((0.5 - 0.25j), (0.25 + 0.5j)),
                                ((-2 + 0.5j), 0.0), (1.0, (-0.25 + 0.5j))])
def test_single_rank_reduces_to_dense_numpy(dtype, op, orders, ab):
    """P = 1, one block: the transform is textbook alpha*op(B) + beta*A on the
    dense matrix.  Power-of-two scalars make every product exact, so numpy and
    the oracle must agree bit for bit whatever the evaluation details.  Complex
    scalars with both parts nonzero (for c128 and c64) reach every term of the
    complex products, alpha's and beta's."""
    alpha, beta = ab
    if dtype not in ("c128", "c64") and (isinstance(alpha, complex) or isinstance(beta, complex)):
        pytest.skip("complex scalars need a complex type")
    M, N = 13, 9
    A = GEN(M, N, [0, M], [0, N], [0], 1, orders[0])
    Bs = GEN(M, N, [0, M], [0, N], [0], 1, orders[1]) if op == "N" else GEN(N, M, [0, N], [0, M], [0], 1, orders[1])
    LA, Ab = _bufs(A, dtype, synth.ROLE_A)
    LB, Bb = _bufs(Bs, dtype, synth.ROLE_B)
    a0 = _dense_from_single_block(Ab[0], A).copy()
    b = _dense_from_single_block(Bb[0], Bs)
    opb = b if op == "N" else (b.T.conj() if op == "C" else b.T)
    nt = oracle.NUMPY[dtype]
    if alpha == 1.0 and beta == 0.0:
        ref = opb.astype(nt)
    elif beta == 0.0:
        ref = (nt(alpha) * opb).astype(nt)
    else:
        ref = (nt(alpha) * opb + nt(beta) * a0).astype(nt)
    oracle.transform(dtype, op, alpha, beta, LA, Ab, LB, Bb)
    got = _dense_from_single_block(Ab[0], A)
    assert np.array_equal(got, ref)


def test_beta_zero_does_not_read_A():
    A = BC(40, 30, 8, 8, 2, 2)
    B = BC(30, 40, 4, 4, 2, 2)
    LA, Ab = _bufs(A, "f64", synth.ROLE_A, fill=False)
    for a in Ab:
        a[:] = np.nan
    LB, Bb = _bufs(B, "f64", synth.ROLE_B)
    oracle.transform("f64", "T", 2.0, 0.0, LA, Ab, LB, Bb)
    assert all(np.isfinite(a).all() for a in Ab)  # every element written, NaN never read


def test_identity_copy_is_a_permutation_of_values():
    w = synth.workload("reshuffle_transpose_1k")
    it = w.items[0]
    LA, Ab = _bufs(it.A, "f64", synth.ROLE_A, fill=False)
    LB, Bb = _bufs(it.B, "f64", synth.ROLE_B)
    oracle.transform("f64", "T", 1.0, 0.0, LA, Ab, LB, Bb)
    a = np.sort(np.concatenate(Ab).view(np.uint64))
    b = np.sort(np.concatenate(Bb).view(np.uint64))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dtype", ["f64", "c128"])
def test_transpose_twice_returns_original(dtype):
    LBs = BC(45, 70, 8, 16, 2, 3, "row", "col")
    LAs = GEN(70, 45, [0, 9, 30, 70], [0, 20, 45], [5, 0, 3, 1, 4, 2], 6, "row")
    LB, Bb = _bufs(LBs, dtype, synth.ROLE_B)
    LA, Ab = _bufs(LAs, dtype, synth.ROLE_A, fill=False)
    op = "C" if dtype == "c128" else "T"
    oracle.transform(dtype, op, 1.0, 0.0, LA, Ab, LB, Bb)
    LB2, Bb2 = _bufs(LBs, dtype, synth.ROLE_B, fill=False)
    oracle.transform(dtype, op, 1.0, 0.0, LB2, Bb2, LA, Ab)
    for x, y in zip(Bb, Bb2):
        assert np.array_equal(x.view(np.uint64), y.view(np.uint64))


def test_conjugate_flips_only_imaginary_sign_bits():
    LBs = BC(33, 21, 5, 4, 2, 2)
    LAs = BC(21, 33, 6, 7, 2, 2, "col", "row")
    LB, Bb = _bufs(LBs, "c128", synth.ROLE_B)
    LA1, A1 = _bufs(LAs, "c128", synth.ROLE_A, fill=False)
    LA2, A2 = _bufs(LAs, "c128", synth.ROLE_A, fill=False)
    oracle.transform("c128", "T", 1.0, 0.0, LA1, A1, LB, Bb)
    oracle.transform("c128", "C", 1.0, 0.0, LA2, A2, LB, Bb)
    for x, y in zip(A1, A2):
        xv, yv = x.view(np.uint64).reshape(-1, 2), y.view(np.uint64).reshape(-1, 2)
        assert np.array_equal(xv[:, 0], yv[:, 0])
        assert np.array_equal(xv[:, 1] ^ yv[:, 1], np.full(xv.shape[0], 1 << 63, np.uint64))


def test_same_layout_identity_is_a_copy():
    spec = BC(50, 44, 7, 5, 3, 2, "col", "row")
    LB, Bb = _bufs(spec, "f64", synth.ROLE_B)
    LA, Ab = _bufs(spec, "f64", synth.ROLE_A, fill=False)
    oracle.transform("f64", "N", 1.0, 0.0, LA, Ab, LB, Bb)
    for x, y in zip(Ab, Bb):
        assert np.array_equal(x, y)


def test_relabeled_target_lands_on_sigma():
    """With sigma, label t's data sits in the buffer of physical rank sigma[t]
    (a 3-cycle, so sigma and its inverse differ)."""
    A = BC(24, 24, 4, 4, 2, 2)
    B = BC(24, 24, 3, 3, 2, 2, "col", "col")
    LB, Bb = _bufs(B, "f64", synth.ROLE_B)
    LA, A_id = _bufs(A, "f64", synth.ROLE_A, fill=False)
    _, A_sg = _bufs(A, "f64", synth.ROLE_A, fill=False)
    sigma = [1, 2, 0, 3]
    oracle.transform("f64", "N", 1.0, 0.0, LA, A_id, LB, Bb)
    oracle.transform("f64", "N", 1.0, 0.0, LA, A_sg, LB, Bb, sigma=sigma)
    for t in range(4):
        assert np.array_equal(A_sg[sigma[t]], A_id[t])


def test_expect_at_matches_full_transform():
    w = synth.workload("scaled_transpose_20k", "small")
    it = w.items[0]
    LB, Bb = _bufs(it.B, "f64", synth.ROLE_B, seed=w.seed)
    LA, Ab = _bufs(it.A, "f64", synth.ROLE_A, seed=w.seed)
    oracle.transform("f64", it.op, it.alpha, it.beta, LA, Ab, LB, Bb)
    rng = np.random.default_rng(0)
    i = rng.integers(0, it.A.nrows, 500)
    j = rng.integers(0, it.A.ncols, 500)
    rank, off, val = oracle.expect_at("f64", it.op, it.alpha, it.beta, LA, LB, None, w.seed, 0, i, j)
    got = np.array([Ab[r][o] for r, o in zip(rank, off)])
    assert np.array_equal(got, val)
    # and one value by hand: A(i,j) = 2*B(j,i) + 0.5*A0(i,j)
    rb, ob = LB.locate(np.array([j[0]]), np.array([i[0]]))
    bval = synth.values("f64", w.seed, synth.stream(synth.ROLE_B, 0, int(rb[0])), 1, int(ob[0]))[0]
    aval = synth.values("f64", w.seed, synth.stream(synth.ROLE_A, 0, int(rank[0])), 1, int(off[0]))[0]
    assert val[0] == 2.0 * bval + 0.5 * aval
