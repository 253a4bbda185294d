"""Pins of the oracle's graph construction and aggregation (CPU only)."""
import numpy as np
import pytest

from oracle import gcn as og
from oracle import graph as gr
from oracle import reduction as rd
from paper_2001_02498_amd import synth


def _fig1(golden):
    g = golden("fig1_aggregation.json")
    e = np.array(g["edges"], dtype=np.int64)
    return g, e[:, 0], e[:, 1]


def test_fig1_neighbour_lists(golden):
    g, s, d = _fig1(golden)
    rp, cl = gr.subgraph_build(g["n"], s, d)
    assert gr.rows_of(rp, cl) == g["neighbours"]


def test_fig1_aggregation_values(golden):
    """Fig. 1 prints the mean-of-neighbours vectors; they are exact."""
    g, s, d = _fig1(golden)
    rp, cl = gr.subgraph_build(g["n"], s, d)
    out = og.aggregate(rp, cl, np.array(g["X"], dtype=np.float64))
    np.testing.assert_array_equal(out, np.array(g["aggregated"], dtype=np.float64))


def test_fig1_reduced_aggregation_values(golden):
    """Aggregating on the reduced graph (Fig. 2 rule applied to Fig. 1)
    reaches the same printed vectors."""
    g, s, d = _fig1(golden)
    rp, cl = gr.subgraph_build(g["n"], s, d)
    red = rd.reduce(rp, cl, theta=1, max_rounds=5)
    assert red["naux"] == 2
    out = og.aggregate_reduced(red, gr.inv_degrees(rp), np.array(g["X"], float))
    np.testing.assert_array_equal(out, np.array(g["aggregated"], dtype=np.float64))


def test_fig2_induced_subgraph(golden):
    g1, s, d = _fig1(golden)
    g2 = golden("fig2_reduction.json")
    rp, cl = gr.subgraph_build(g1["n"], s, d, vertices=g2["subset"])
    assert gr.rows_of(rp, cl) == g2["neighbours_before"]


def test_induced_subgraph_relabels_in_given_order():
    # path 0-1-2-3; subset [3, 1, 2] -> 3->0, 1->1, 2->2; edges 1-2, 2-3 survive
    rp, cl = gr.subgraph_build(4, [0, 1, 2], [1, 2, 3], vertices=[3, 1, 2])
    assert gr.rows_of(rp, cl) == [[2], [2], [0, 1]]


def test_build_against_brute_force_sets():
    rng = np.random.default_rng(7)
    for trial in range(20):
        n = int(rng.integers(1, 40))
        s, d = synth.random_edges(n, int(rng.integers(0, 4 * n)), rng)
        rp, cl = gr.subgraph_build(n, s, d)
        want = [set() for _ in range(n)]
        for a, b in zip(s, d):
            if a != b:
                want[a].add(int(b))
                want[b].add(int(a))
        assert gr.rows_of(rp, cl) == [sorted(x) for x in want]
        A = gr.adjacency_dense(rp, cl)
        assert np.array_equal(A, A.T)
        assert np.all(np.diag(A) == 0)
        assert A.max(initial=0) <= 1


def test_build_rejects_bad_input():
    with pytest.raises(gr.GraphError):
        gr.subgraph_build(3, [0, 5], [1, 2])
    with pytest.raises(gr.GraphError):
        gr.subgraph_build(3, [0], [1], vertices=[0, 0])
    with pytest.raises(gr.GraphError):
        gr.subgraph_build(3, [0, 1], [1])


def test_aggregation_equals_dense_definition():
    """D^-1 A H against the textbook dense product built from the edge set."""
    rng = np.random.default_rng(3)
    for trial in range(10):
        n = int(rng.integers(2, 30))
        s, d = synth.random_edges(n, 3 * n, rng)
        rp, cl = gr.subgraph_build(n, s, d)
        A = np.zeros((n, n))
        for a, b in zip(s, d):
            if a != b:
                A[a, b] = A[b, a] = 1.0
        deg = A.sum(1)
        Dinv = np.diag([1.0 / x if x else 0.0 for x in deg])
        H = rng.standard_normal((n, 5))
        np.testing.assert_allclose(og.aggregate(rp, cl, H), Dinv @ A @ H,
                                   rtol=1e-13, atol=1e-13)
        G = rng.standard_normal((n, 4))
        np.testing.assert_allclose(og.aggregate_transposed(rp, cl, G),
                                   A @ Dinv @ G, rtol=1e-13, atol=1e-13)
        # the transposed form is the transpose of the forward operator
        np.testing.assert_allclose(A @ Dinv, (Dinv @ A).T)


def test_constant_features_stay_constant():
    """Rows of D^-1 A sum to one: constant features aggregate to themselves
    (and isolated vertices to zero)."""
    wl = synth.small_workload(300, 6, 2, 8, 4, 3, synth.SOFTMAX_CE, (1,))
    inp = synth.make_inputs(wl)
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    H = np.full((wl.n, 7), 2.5)
    out = og.aggregate(rp, cl, H)
    deg = gr.degrees(rp)
    assert np.all(out[deg > 0] == 2.5)
    assert np.all(out[deg == 0] == 0.0)
