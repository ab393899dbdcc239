"""Relabeling variants (host only): the paper's greedy 2-approximation and the
latency-bandwidth topology cost of Section 3, library vs oracle."""
import itertools

import numpy as np
import pytest

import oracle

C = pytest.importorskip("paper_2106_06601_amd")


def _rand(rng, P, hi=6, zero=0.3):
    V = rng.integers(0, hi, size=(P, P)).astype(np.int64)
    V[rng.random((P, P)) < zero] = 0
    return V


def test_greedy_locally_free_matches_oracle():
    rng = np.random.default_rng(21)
    for P in list(range(1, 10)) + [16, 33]:
        for _ in range(3):
            V = _rand(rng, P, hi=5)
            sig, before, after = C.costa_relabel_cost(V, method="greedy")
            assert sig == oracle.relabel_greedy(V)
            assert before == oracle.total_cost(V, list(range(P)))
            assert after == oracle.total_cost(V, sig)


def test_greedy_never_raises_the_cost():
    """Gains can be negative: on [[7, 2], [0, 0]] the greedy perfect matching
    has total gain -5 and the identity is kept (both costs)."""
    V = np.array([[7, 2], [0, 0]], np.int64)
    assert C.costa_relabel_cost(V, method="greedy") == ([0, 1], 2.0, 2.0)  # only V[0][1] is remote
    L = np.array([[0.0, 1.0], [1.0, 0.0]])
    Bw = np.array([[0.0, 1.0], [1.0, 0.0]])
    sig, before, after = C.costa_relabel_cost(V, 1.0, L, Bw, "greedy")
    assert sig == [0, 1] and before == after == 3.0
    rng = np.random.default_rng(23)
    for P in (2, 3, 5, 8, 17):
        for _ in range(5):
            V = _rand(rng, P, hi=9, zero=0.1)
            _, before, after = C.costa_relabel_cost(V, method="greedy")
            assert after <= before
            L = rng.random((P, P))
            Bw = rng.random((P, P))
            np.fill_diagonal(L, 0.0)
            np.fill_diagonal(Bw, 0.0)
            _, before, after = C.costa_relabel_cost(V, 4.0, L, Bw, "greedy")
            assert after <= before


def test_exact_locally_free_is_the_canonical_relabeling():
    rng = np.random.default_rng(22)
    for P in (3, 7, 12):
        V = _rand(rng, P, hi=4)
        sig, before, after = C.costa_relabel_cost(V, elem_bytes=8.0)
        assert sig == C.costa_relabel(V)[0] == oracle.relabel(V)
        # cost in bytes: remote elements x 8
        assert after == 8 * oracle.total_cost(V, sig)
        assert before == 8 * oracle.total_cost(V, list(range(P)))


def _topology(P, nodes, lat_inter, bw_intra, bw_inter, rng=None):
    node = [r * nodes // P for r in range(P)]
    L = np.zeros((P, P))
    B = np.zeros((P, P))
    for i in range(P):
        for j in range(P):
            same = node[i] == node[j]
            L[i, j] = 0.0 if same else lat_inter
            B[i, j] = (0.0 if i == j else bw_intra) if same else bw_inter
            if rng is not None and not same:
                B[i, j] += float(rng.integers(0, 3))
    return L, B


def test_exact_topology_cost_matches_bruteforce():
    rng = np.random.default_rng(23)
    for P in range(2, 8):
        for _ in range(3):
            V = _rand(rng, P, hi=20)
            L, B = _topology(P, 2, 5.0, 1.0, 4.0, rng)
            w = oracle.w_topology(L, B, 8.0)
            ref = oracle.relabel_bruteforce_cost(V, w)
            sig, before, after = C.costa_relabel_cost(V, 8.0, L, B, "exact")
            assert sorted(sig) == list(range(P))
            assert after == pytest.approx(oracle.total_cost(V, sig, w), rel=1e-12)
            assert after == pytest.approx(oracle.total_cost(V, ref, w), rel=1e-12)  # optimal
            assert before == pytest.approx(oracle.total_cost(V, list(range(P)), w), rel=1e-12)


def test_greedy_topology_cost_matches_oracle_and_two_approximation():
    rng = np.random.default_rng(24)
    for P in range(2, 9):
        for _ in range(3):
            V = _rand(rng, P, hi=20)
            L, B = _topology(P, 2, 3.0, 1.0, 5.0)
            w = oracle.w_topology(L, B, 1.0)
            sig, before, after = C.costa_relabel_cost(V, 1.0, L, B, "greedy")
            assert sig == oracle.relabel_greedy(V, w)
            # greedy matching on non-negative weights is a 2-approximation; the
            # gains shifted by their minimum are non-negative and keep the order
            gains = np.array([[oracle.gain(V, x, y, w) for y in range(P)] for x in range(P)], dtype=float)
            shift = gains - gains.min()
            opt = oracle.relabel_bruteforce_cost(V, w)
            g_greedy = sum(shift[x, sig[x]] for x in range(P))
            g_opt = sum(shift[x, opt[x]] for x in range(P))
            assert g_greedy >= g_opt / 2 - 1e-9


def test_topology_cost_hand_example():
    """P = 2: rank 0 sends 5 elements to label 1, rank 1 sends 3 to label 0;
    latency 2 and 1 unit per byte between the ranks, nothing within a rank.
    Identity: w(0,1,5) + w(1,0,3) = (2 + 5) + (2 + 3) = 12.  Swapping the labels
    makes both packages local: W = 0.  Gains by eq:delta: delta(p_0, p_1) =
    w(1,0,3) - w(1,1,3) = 5, delta(p_1, p_0) = w(0,1,5) - w(0,0,5) = 7."""
    V = np.array([[0, 5], [3, 0]], np.int64)
    L = np.array([[0.0, 2.0], [2.0, 0.0]])
    B = np.array([[0.0, 1.0], [1.0, 0.0]])
    w = oracle.w_topology(L, B, 1.0)
    assert oracle.gain(V, 0, 1, w) == 5 and oracle.gain(V, 1, 0, w) == 7
    for method in ("exact", "greedy"):
        sig, before, after = C.costa_relabel_cost(V, 1.0, L, B, method)
        assert (sig, before, after) == ([1, 0], 12.0, 0.0)


def test_relabel_cost_errors():
    V = np.ones((2, 2), np.int64)
    with pytest.raises(C.CostaError):
        C.costa_relabel_cost(V, 1.0, np.zeros((2, 2)), None)
    with pytest.raises(C.CostaError):
        C.costa_relabel_cost(V, 1.0, -np.ones((2, 2)), np.ones((2, 2)))
    with pytest.raises(C.CostaError):
        C.costa_relabel_cost(V, 0.0)
