"""Pins of the oracle's redundancy reduction (Algorithms 1-3, Theorem 1)."""
import collections

import networkx as nx
import numpy as np
import pytest
import scipy.sparse as sp

from oracle import gcn as og
from oracle import graph as gr
from oracle import reduction as rd
from paper_2001_02498_amd import synth


def _fig2(golden):
    g1 = golden("fig1_aggregation.json")
    g2 = golden("fig2_reduction.json")
    e = np.array(g1["edges"])
    rp, cl = gr.subgraph_build(g1["n"], e[:, 0], e[:, 1], vertices=g2["subset"])
    return g2, rp, cl


def _random_graph(rng, n, m):
    s, d = synth.random_edges(n, m, rng)
    return gr.subgraph_build(n, s, d)


def test_fig2_aggregation_graph(golden):
    g2, rp, cl = _fig2(golden)
    W, D = rd.aggregation_graph_literal(gr.rows_of(rp, cl))
    assert sorted([a, b, w] for (a, b), w in W.items()) == g2["aggregation_graph"]
    # attribute sets: lists holding both endpoints
    assert D[(0, 2)] == {1, 3} and D[(1, 3)] == {0, 2}


def test_fig2_reduction_exact(golden):
    g2, rp, cl = _fig2(golden)
    red = rd.reduce(rp, cl, theta=g2["theta"], max_rounds=5)
    assert red["pairs"].tolist() == g2["pairs"]
    assert red["round_offsets"].tolist() == g2["round_offsets"]
    assert red["rowptr"].tolist() == g2["rowptr"]
    assert red["col"].tolist() == g2["col"]
    rows0 = gr.rows_of(rp, cl)
    rows1 = gr.rows_of(red["rowptr"], red["col"])
    assert rd.num_read(rows0) == g2["num_read_before"]
    assert rd.num_add(rows0) == g2["num_add_before"]
    assert rd.num_read(rows1) == g2["num_read_after"]
    assert rd.num_add(rows1) == g2["num_add_after"]
    gread, gadd = rd.gammas(rp, cl, red)
    assert gread == pytest.approx(g2["gamma_read"])
    assert gadd == pytest.approx(g2["gamma_add"])


def test_fig1_reduction_exact(golden):
    g1 = golden("fig1_aggregation.json")
    want = golden("fig1_reduction.json")
    e = np.array(g1["edges"])
    rp, cl = gr.subgraph_build(g1["n"], e[:, 0], e[:, 1])
    for literal in (False, True):
        red = rd.reduce(rp, cl, theta=1, literal=literal)
        assert red["pairs"].tolist() == want["pairs"]
        assert red["round_offsets"].tolist() == want["round_offsets"]
        assert red["rowptr"].tolist() == want["rowptr"]
        assert red["col"].tolist() == want["col"]
        assert red["stats"][0][2] == want["num_read_after"]
        assert red["stats"][0][3] == want["num_add_after"]


def test_threshold_two_leaves_figures_unchanged(golden):
    g2, rp, cl = _fig2(golden)
    red = rd.reduce(rp, cl, theta=2)
    assert red["naux"] == 0
    assert red["rowptr"].tolist() == rp.tolist() and red["col"].tolist() == cl.tolist()


def test_pair_weights_match_sparse_product():
    """Alg. 1 weight of {x, y} = number of lists holding both = (M^T M)[x, y]
    with M the aggregator-by-vertex 0/1 matrix."""
    rng = np.random.default_rng(11)
    for trial in range(15):
        n = int(rng.integers(3, 60))
        rp, cl = _random_graph(rng, n, 4 * n)
        M = sp.csr_matrix((np.ones(cl.size), cl, rp), shape=(n, n))
        P = (M.T @ M).tocoo()
        want = {(int(a), int(b)): int(v) for a, b, v in zip(P.row, P.col, P.data)
                if a < b and v >= 2}
        x, y, w = rd.pair_weights(gr.rows_of(rp, cl), n)
        got = {(int(a), int(b)): int(c) for a, b, c in zip(x, y, w)}
        assert got == want
        lit, _ = rd.aggregation_graph_literal(gr.rows_of(rp, cl))
        assert lit == want


def test_literal_and_vectorised_reduction_agree():
    rng = np.random.default_rng(5)
    for trial in range(10):
        n = int(rng.integers(5, 50))
        rp, cl = _random_graph(rng, n, 5 * n)
        for theta in (1, 2):
            a = rd.reduce(rp, cl, theta=theta, max_rounds=4)
            b = rd.reduce(rp, cl, theta=theta, max_rounds=4, literal=True)
            for k in ("rowptr", "col", "pairs", "round_offsets"):
                assert np.array_equal(a[k], b[k])


def test_theorem1_exact_per_round():
    """Each matched pair of weight W removes exactly W list entries (and W
    additions): the counts fall by sum(W) per round; with the two reads and
    one addition of each pre-sum, reads fall by sum(W - 2), additions by
    sum(W - 1) (Theorem 1)."""
    wl = synth.small_workload(400, 12, 2, 4, 4, 2, synth.SOFTMAX_CE, (2,))
    inp = synth.make_inputs(wl)
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    rows0 = gr.rows_of(rp, cl)
    red = rd.reduce(rp, cl, theta=2, max_rounds=5)
    assert len(red["stats"]) >= 2
    prev_read, prev_add = rd.num_read(rows0), rd.num_add(rows0)
    for (m, wsum, nread, nadd) in red["stats"]:
        assert nread == prev_read - wsum
        assert nadd == prev_add - wsum
        assert (prev_read - nread) - 2 * m == wsum - 2 * m   # sum(W - 2)
        prev_read, prev_add = nread, nadd


def test_expansion_invariant_and_structure():
    """Expanding the new ids of each reduced list gives back N(w), each
    neighbour exactly once; lists are sorted; ids of a round only use
    earlier ids."""
    rng = np.random.default_rng(9)
    for trial in range(8):
        n = int(rng.integers(20, 120))
        rp, cl = _random_graph(rng, n, 8 * n)
        red = rd.reduce(rp, cl, theta=2, max_rounds=5)
        pairs, off = red["pairs"], red["round_offsets"]
        for r in range(len(off) - 1):
            for k in range(off[r], off[r + 1]):
                a, b = pairs[k]
                assert a < b < n + off[r]
        rows0 = gr.rows_of(rp, cl)
        rows1 = gr.rows_of(red["rowptr"], red["col"])
        for w in range(n):
            assert rows1[w] == sorted(rows1[w])
            exp = []
            for c in rows1[w]:
                exp += rd.expand(c, n, pairs)
            assert collections.Counter(exp) == collections.Counter(rows0[w])


def test_greedy_is_maximal_and_half_approximate():
    rng = np.random.default_rng(13)
    for trial in range(25):
        n = int(rng.integers(6, 18))
        rp, cl = _random_graph(rng, n, 5 * n)
        rows = gr.rows_of(rp, cl)
        x, y, w = rd.pair_weights(rows, n)
        for theta in (1, 2):
            got, _ = rd.greedy_matching(x, y, w, theta, n)
            used = set()
            for a, b, _ in got:
                assert a not in used and b not in used
                used |= {a, b}
            cand = [(int(a), int(b), int(c)) for a, b, c in zip(x, y, w) if c > theta]
            for a, b, _ in cand:          # maximal among candidates
                assert a in used or b in used
            G = nx.Graph()
            for a, b, c in cand:
                G.add_edge(a, b, weight=c)
            best = nx.max_weight_matching(G)
            best_w = sum(G[a][b]["weight"] for a, b in best)
            got_w = sum(c for _, _, c in got)
            assert 2 * got_w >= best_w


def test_greedy_tie_break_order():
    # equal weights: smaller first id, then smaller second id wins
    x = np.array([0, 0, 1], dtype=np.int64)
    y = np.array([2, 1, 2], dtype=np.int64)
    w = np.array([3, 3, 3], dtype=np.int64)
    got, _ = rd.greedy_matching(x, y, w, 2, 3)
    assert got == [(0, 1, 3)]
    # heavier pair first regardless of ids
    w = np.array([3, 3, 5], dtype=np.int64)
    got, _ = rd.greedy_matching(x, y, w, 2, 3)
    assert got == [(1, 2, 5)]


def test_budget_caps_new_vertices():
    wl = synth.small_workload(300, 12, 2, 4, 4, 2, synth.SOFTMAX_CE, (3,))
    inp = synth.make_inputs(wl)
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    full = rd.reduce(rp, cl, theta=2, max_rounds=5)
    assert full["naux"] > 10
    cap = full["naux"] // 3
    red = rd.reduce(rp, cl, theta=2, max_rounds=5, max_aux=cap)
    assert red["naux"] == cap
    # the capped result is a prefix of the uncapped one
    assert np.array_equal(red["pairs"], full["pairs"][:cap])
    none = rd.reduce(rp, cl, theta=2, max_rounds=5, max_aux=0)
    assert none["naux"] == 0 and np.array_equal(none["col"], cl)


def test_zero_rounds_is_identity():
    rng = np.random.default_rng(2)
    rp, cl = _random_graph(rng, 30, 100)
    red = rd.reduce(rp, cl, max_rounds=0)
    assert red["naux"] == 0
    assert np.array_equal(red["rowptr"], rp) and np.array_equal(red["col"], cl)


def test_direct_equals_reduced_aggregation():
    """The reduced graph reaches D^-1 A H exactly for integer features (all
    partial sums exact), and to rounding for real ones; likewise the
    transposed form with the degree scaling moved in front."""
    wl = synth.small_workload(500, 14, 2, 4, 4, 2, synth.SOFTMAX_CE, (4,))
    inp = synth.make_inputs(wl)
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    red = rd.reduce(rp, cl, theta=2, max_rounds=5)
    assert red["naux"] > 0
    inv = gr.inv_degrees(rp)
    rng = np.random.default_rng(0)
    Hi = rng.integers(-50, 50, size=(wl.n, 6)).astype(np.float64)
    A = og.adjacency(rp, cl, wl.n)
    np.testing.assert_array_equal(og.aggregate_reduced(red, inv, Hi, "post") / 1.0,
                                  inv[:, None] * (A @ Hi))
    Hr = rng.standard_normal((wl.n, 6))
    np.testing.assert_allclose(og.aggregate_reduced(red, inv, Hr, "post"),
                               og.aggregate(rp, cl, Hr), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(og.aggregate_reduced(red, inv, Hr, "pre"),
                               og.aggregate_transposed(rp, cl, Hr),
                               rtol=1e-12, atol=1e-12)
