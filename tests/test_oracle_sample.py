"""Pins of the oracle's frontier sampler and induced subgraph
(Section 3.1; the sampler is the cited multi-dimensional random walk).

Each check rests on something other than the oracle's own code: the
generator's published outputs, the structure of a single random walk, a
closed-form step share between two regular components, uniform neighbour
choice, the cited method's steady state (visits in proportion to degree),
and brute force over a dense adjacency matrix."""
import itertools

import numpy as np
import pytest

from oracle import graph as ograph
from oracle import sample as osample


def _csr(n, edges):
    src = [a for a, _ in edges]
    dst = [b for _, b in edges]
    rp, cl = ograph.subgraph_build(n, src, dst)
    return [int(x) for x in rp], [int(x) for x in cl]


def _random_edges(rng, n, m):
    a = rng.integers(0, n, m)
    b = rng.integers(0, n, m)
    return [(int(x), int(y)) for x, y in zip(a, b)]


def test_splitmix64_published_outputs(golden):
    fx = golden("splitmix64_outputs.json")
    for seq in fx["sequences"]:
        got = [osample.splitmix64(seq["seed"], i) for i in range(len(seq["outputs"]))]
        assert got == [int(x) for x in seq["outputs"]]


def test_bounded_draws():
    # a power-of-two bound keeps the output's top bits exactly
    d = osample.Draws(99)
    for i in range(50):
        assert d.below(1 << 12) == osample.splitmix64(99, i) >> 52
    # bound 1 always gives 0; other bounds stay in range and are uniform
    assert all(osample.Draws(5).below(1) == 0 for _ in range(10))
    d = osample.Draws(7)
    counts = np.bincount([d.below(7) for _ in range(70000)], minlength=7)
    assert counts.size == 7
    chi2 = ((counts - 10000) ** 2 / 10000).sum()
    assert chi2 < 30.0     # 6 degrees of freedom; p ~ 4e-5 at 30


def test_single_walker_is_a_random_walk():
    rng = np.random.default_rng(3)
    n = 60
    rp, cl = _csr(n, _random_edges(rng, n, 240))
    trace = []
    osample.frontier_sample(rp, cl, 1, n, seed=11, max_steps=400, trace=trace)
    assert trace
    for t, (slot, u, v) in enumerate(trace):
        assert slot == 0
        assert v in cl[rp[u]:rp[u + 1]]
        if t:
            assert u == trace[t - 1][2]


def test_degree_weighted_pick_between_components():
    # K_11 (degree 10) and a 2000-cycle (degree 2), one walker in each: every
    # step has frontier degree sum 12, so the clique walker moves with
    # probability 10/12 exactly (a uniform pick would give 1/2)
    k, c = 11, 2000
    edges = [(a, b) for a, b in itertools.combinations(range(k), 2)]
    edges += [(k + i, k + (i + 1) % c) for i in range(c)]
    n = k + c
    rp, cl = _csr(n, edges)
    seed = next(s for s in range(1000)
                if (lambda f: (f[0] < k) != (f[1] < k))(
                    osample.frontier_sample(rp, cl, 2, n, seed=s, max_steps=0)))
    trace = []
    steps = 20000
    osample.frontier_sample(rp, cl, 2, n, seed=seed, max_steps=steps, trace=trace)
    assert len(trace) == steps
    share = sum(1 for _, u, _ in trace if u < k) / steps
    assert abs(share - 10 / 12) < 0.012     # ~4.5 standard deviations


def test_neighbour_choice_uniform():
    # star: the walker alternates centre -> leaf, each leaf equally likely
    leaves = 9
    rp, cl = _csr(leaves + 1, [(0, i) for i in range(1, leaves + 1)])
    trace = []
    osample.frontier_sample(rp, cl, 1, leaves + 1, seed=5, max_steps=20000, trace=trace)
    from_centre = [v for _, u, v in trace if u == 0]
    assert all(v != 0 for v in from_centre)
    assert all(v == 0 for _, u, v in trace if u != 0)
    counts = np.bincount(from_centre, minlength=leaves + 1)[1:]
    expect = len(from_centre) / leaves
    chi2 = ((counts - expect) ** 2 / expect).sum()
    assert chi2 < 30.0     # 8 degrees of freedom


def test_visits_follow_degree_in_steady_state():
    # the cited method's steady state samples every edge equally often, so
    # the vertex a step lands on is drawn in proportion to its degree. 100
    # isolated vertices keep the budget (all n vertices) out of reach, so the
    # walk runs for max_steps; the seed puts two walkers in the component
    edges = [(a, b) for a, b in itertools.combinations(range(5), 2)]       # K_5
    edges += [(4, 5), (5, 6), (6, 7), (7, 8), (8, 9), (9, 7), (2, 9), (1, 6)]
    core, n = 10, 110
    rp, cl = _csr(n, edges)
    seed = next(s for s in range(100000)
                if sum(v < core for v in
                       osample.frontier_sample(rp, cl, 3, n, seed=s, max_steps=0)) >= 2)
    trace = []
    steps = 100000
    osample.frontier_sample(rp, cl, 3, n, seed=seed, max_steps=steps, trace=trace)
    assert len(trace) == steps
    deg = np.diff(rp)[:core]
    visits = np.bincount([v for _, _, v in trace], minlength=core) / steps
    tv = 0.5 * np.abs(visits - deg / deg.sum()).sum()
    assert tv < 0.02


def test_initial_frontier_uniform_and_distinct():
    rng = np.random.default_rng(1)
    n, m = 20, 5
    rp, cl = _csr(n, _random_edges(rng, n, 60))
    hits = np.zeros(n)
    runs = 2000
    for s in range(runs):
        f = osample.frontier_sample(rp, cl, m, m, seed=s, max_steps=0)
        assert len(f) == m == len(set(f))
        hits[f] += 1
    assert np.abs(hits / runs - m / n).max() < 0.05


def test_stopping_rules():
    rng = np.random.default_rng(2)
    n = 200
    edges = [(i, i + 1) for i in range(n - 1)] + _random_edges(rng, n, 600)
    rp, cl = _csr(n, edges)          # connected (contains a path)
    for budget in (7, 50, 200):
        got = osample.frontier_sample(rp, cl, 4, budget, seed=budget, max_steps=10 ** 6)
        assert len(got) == budget
        assert got == sorted(set(got)) and 0 <= got[0] and got[-1] < n
    # the walk cap: no steps leaves the initial frontier
    assert len(osample.frontier_sample(rp, cl, 4, 50, seed=1, max_steps=0)) == 4
    # a frontier of isolated vertices cannot move
    rp0, cl0 = _csr(30, [])
    assert len(osample.frontier_sample(rp0, cl0, 6, 30, seed=3, max_steps=100)) == 6
    with pytest.raises(ValueError):
        osample.frontier_sample(rp, cl, 5, 4, seed=0, max_steps=1)
    with pytest.raises(ValueError):
        osample.frontier_sample(rp, cl, 1, n + 1, seed=0, max_steps=1)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_induce_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = 30
    edges = _random_edges(rng, n, 90)
    rp, cl = _csr(n, edges)
    A = np.zeros((n, n), dtype=np.int64)
    for a, b in edges:
        if a != b:
            A[a, b] = A[b, a] = 1
    V = rng.permutation(n)[:17]
    sub = A[np.ix_(V, V)]
    irp, icl = osample.induce(rp, cl, V)
    assert irp[-1] == sub.sum()
    for k in range(len(V)):
        assert list(icl[irp[k]:irp[k + 1]]) == list(np.flatnonzero(sub[k]))
