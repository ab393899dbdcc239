"""Relabeling on device volume matrices (GPU): the five workloads and random
layouts, every method and cost of costa_relabel_cost against the oracle.

The volume matrix comes from the device (costa_volume_matrix) and is first
checked against the oracle's count; the relabelings are then compared with
the oracle's: the canonical exact relabeling and the greedy matching under
the locally-free cost (Section 4, Section 6), and both under the
latency-bandwidth topology cost of Section 3 (brute force for P <= 7, else
the optimal total gain of the eq:delta gains from an assignment solver).
"""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2106_06601_amd as C


def _say(msg):
    print(msg, flush=True)


def _topology(P, per_node=8, lat=5.0, inv_bw_intra=1.0, inv_bw_inter=8.0):
    """Ranks grouped in nodes of `per_node`: nothing within a rank, a cheap
    link within a node, latency plus a slow link between nodes."""
    node = np.arange(P) // per_node
    same = node[:, None] == node[None, :]
    L = np.where(same, 0.0, lat)
    B = np.where(same, inv_bw_intra, inv_bw_inter)
    np.fill_diagonal(B, 0.0)
    return L, B


def _max_total_gain(V, w):
    from scipy.optimize import linear_sum_assignment
    P = V.shape[0]
    G = np.array([[oracle.gain(V, x, y, w) for y in range(P)] for x in range(P)], dtype=float)
    r, c = linear_sum_assignment(G, maximize=True)
    return G[r, c].sum()


def _check_all(V):
    P = V.shape[0]
    ident = list(range(P))
    # locally-free cost: exact (canonical) and greedy
    sig, before, after = C.costa_relabel_cost(V, method="exact")
    assert sig == oracle.relabel(V) == C.costa_relabel(V)[0]
    assert before == oracle.total_cost(V, ident) and after == oracle.total_cost(V, sig)
    sig_g, before_g, after_g = C.costa_relabel_cost(V, method="greedy")
    assert sig_g == oracle.relabel_greedy(V)
    assert before_g == before and after_g == oracle.total_cost(V, sig_g)
    assert after <= after_g <= before
    # topology cost (8-byte elements)
    L, B = _topology(P)
    w = oracle.w_topology(L, B, 8.0)
    sig, before, after = C.costa_relabel_cost(V, 8.0, L, B, "exact")
    assert sorted(sig) == ident
    assert before == pytest.approx(oracle.total_cost(V, ident, w), rel=1e-12)
    assert after == pytest.approx(oracle.total_cost(V, sig, w), rel=1e-12)
    if P <= 7:
        assert after == pytest.approx(oracle.total_cost(V, oracle.relabel_bruteforce_cost(V, w), w), rel=1e-12)
    else:
        # Lemma 2: W(G_sigma) = W(G) - Delta_sigma, so the optimum removes the
        # largest total gain an assignment can reach
        best = _max_total_gain(V, w)
        assert oracle.total_gain(V, sig, w) == pytest.approx(best, rel=1e-9, abs=1e-6)
        assert after == pytest.approx(before - best, rel=1e-9, abs=1e-6)
    sig_g, _, after_g = C.costa_relabel_cost(V, 8.0, L, B, "greedy")
    assert sig_g == oracle.relabel_greedy(V, w)
    assert after_g == pytest.approx(oracle.total_cost(V, sig_g, w), rel=1e-12)
    assert after <= after_g * (1 + 1e-12) and after_g <= before * (1 + 1e-12)


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_relabel_variants_on_device_volumes(name):
    w = synth.workload(name)
    _say(f"relabeling variants: {name}")
    V = None
    for it in w.items:
        v = C.costa_volume_matrix(C.layout_from_spec(it.A), C.layout_from_spec(it.B), it.op)
        if name != "rpa_batched_tall_skinny":  # its closed form is checked in test_gpu_parity
            assert np.array_equal(v, oracle.volume(oracle.OLayout(it.A), oracle.OLayout(it.B), it.op))
        V = v if V is None else V + v
    _check_all(V)


@pytest.mark.parametrize("P", [3, 6, 8, 16, 33, 64])
def test_relabel_variants_on_random_layouts(P):
    for seed in range(2):
        A, B = synth.random_layout_pair(P, 100 * P + seed, n=1024)
        _say(f"relabeling variants: random layouts P={P} seed={seed}")
        V = C.costa_volume_matrix(C.layout_from_spec(A), C.layout_from_spec(B), "N")
        assert np.array_equal(V, oracle.volume(oracle.OLayout(A), oracle.OLayout(B), "N"))
        _check_all(V)
