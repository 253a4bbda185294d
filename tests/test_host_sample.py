"""The library's frontier sampler and induced subgraph (host C++) against the
oracle (Section 3.1: a minibatch is the subgraph induced on vertices that a
graph sampler draws; the sampler is the cited multi-dimensional random
walk). Integer results, so every comparison is exact: the sampled ids, the
number of steps, and the induced CSR; also the pipeline's sampled jobs."""
import ctypes

import numpy as np
import pytest

from oracle import graph as ograph
from oracle import reduction as ored
from oracle import sample as osample
from paper_2001_02498_amd import synth

gcn = pytest.importorskip("paper_2001_02498_amd.gcn")


def _graphs(seed, n, m_edges, isolated=0):
    """Random multigraph edge list with `isolated` extra vertices no edge touches."""
    rng = np.random.default_rng(seed)
    s, d = synth.random_edges(n, m_edges, rng)
    return n + isolated, s, d


def _oracle_csr(n, s, d):
    rp, cl = ograph.subgraph_build(n, s, d)
    return [int(x) for x in rp], [int(x) for x in cl]


def _oracle_sample(rp, cl, m, budget, seed, max_steps):
    trace = []
    got = osample.frontier_sample(rp, cl, m, budget, seed, max_steps, trace=trace)
    return np.asarray(got, dtype=np.int32), len(trace)


@pytest.mark.parametrize("case", [
    # (graph seed, n, edges, isolated, m, budget, sample seed, max_steps)
    (0, 50, 150, 0, 1, 30, 7, 10 ** 6),
    (1, 200, 900, 5, 5, 120, 123, 10 ** 6),
    (2, 300, 600, 40, 17, 250, 2 ** 64 - 1, 10 ** 6),
    (3, 400, 3000, 0, 50, 400, 99, 10 ** 6),        # budget = n
    (4, 400, 3000, 0, 50, 300, 5, 40),              # stopped by max_steps
    (5, 120, 80, 30, 8, 100, 11, 10 ** 6),          # sparse, walkers strand
    (6, 64, 2000, 0, 64, 64, 3, 10 ** 6),           # m = budget: no steps
])
def test_sample_matches_oracle(case):
    gseed, n, ne, iso, m, budget, seed, max_steps = case
    n, s, d = _graphs(gseed, n, ne, iso)
    full = gcn.subgraph_build(n, s, d)
    rp, cl = _oracle_csr(n, s, d)
    want, want_steps = _oracle_sample(rp, cl, m, budget, seed, max_steps)
    got, steps = gcn.sample_frontier(full, m, budget, seed, max_steps)
    assert steps == want_steps
    assert np.array_equal(got, want)


def test_sample_power_law_full_graph():
    # the full-graph generator's structure (hubs, isolated vertices) at a
    # size the plain-loop oracle walks in seconds
    wl = synth.SAMPLED["yelpfull"]
    fi = synth.make_full_inputs(wl, n_full=20000)
    full = gcn.subgraph_build(20000, fi.src, fi.dst)
    rp, cl = (np.asarray(a) for a in full.csr())
    orp, ocl = ograph.subgraph_build(20000, fi.src, fi.dst)
    assert np.array_equal(rp, orp) and np.array_equal(cl, ocl)
    rp, cl = [int(x) for x in orp], [int(x) for x in ocl]
    for i in range(2):
        seed = wl.sample_seed(i)
        want, want_steps = _oracle_sample(rp, cl, 40, 1500, seed, wl.max_steps)
        got, steps = gcn.sample_frontier(full, 40, 1500, seed, wl.max_steps)
        assert steps == want_steps and np.array_equal(got, want)
        assert got.size == 1500


def test_sample_edge_cases():
    # edgeless graph: the frontier cannot move
    full = gcn.subgraph_build(30, [], [])
    got, steps = gcn.sample_frontier(full, 6, 30, 3, 100)
    want, _ = _oracle_sample([0] * 31, [], 6, 30, 3, 100)
    assert steps == 0 and np.array_equal(got, want) and got.size == 6
    # max_steps = 0 leaves the initial frontier
    n, s, d = _graphs(8, 100, 500)
    full = gcn.subgraph_build(n, s, d)
    got, steps = gcn.sample_frontier(full, 9, 50, 1, 0)
    assert steps == 0 and got.size == 9
    # a single vertex
    one = gcn.subgraph_build(1, [], [])
    got, steps = gcn.sample_frontier(one, 1, 1, 0, 10)
    assert list(got) == [0] and steps == 0


@pytest.mark.parametrize("m,budget,steps", [(0, 5, 1), (6, 5, 1), (1, 101, 1), (1, 5, -1)])
def test_sample_rejects(m, budget, steps):
    n, s, d = _graphs(9, 100, 300)
    full = gcn.subgraph_build(n, s, d)
    with pytest.raises(gcn.GcnError) as e:
        gcn.sample_frontier(full, m, budget, 0, steps)
    assert e.value.code == gcn.E_INVALID_ARG


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_induce_matches_oracle_and_build(seed):
    rng = np.random.default_rng(seed)
    n, s, d = _graphs(seed + 20, 400, 2500, 10)
    full = gcn.subgraph_build(n, s, d)
    rp, cl = ograph.subgraph_build(n, s, d)
    for V in (np.sort(rng.choice(n, 150, replace=False)),     # ascending (sampler order)
              rng.permutation(n)[:150],                        # any order
              np.arange(n), np.zeros(0, np.int64)):
        sub = gcn.subgraph_induce(full, V)
        grp, gcl = sub.csr()
        orp, ocl = osample.induce(rp, cl, V)
        assert np.array_equal(grp, orp) and np.array_equal(gcl, ocl)
        brp, bcl = gcn.subgraph_build(n, s, d, vertices=V).csr()
        assert np.array_equal(grp, brp) and np.array_equal(gcl, bcl)


def test_induce_rejects():
    n, s, d = _graphs(30, 50, 200)
    full = gcn.subgraph_build(n, s, d)
    for V in ([1, 2, 1], [0, 50], [-1]):
        with pytest.raises(gcn.GcnError) as e:
            gcn.subgraph_induce(full, V)
        assert e.value.code == gcn.E_INVALID_ARG


def _image(ptr, nb):
    return np.frombuffer((ctypes.c_uint8 * nb).from_address(ptr), dtype=np.uint8).copy()


@pytest.mark.parametrize("workers", [1, 4])
def test_pipeline_sampled_jobs(workers):
    # each sampled job = the oracle's walk, the induced subgraph, the reduced
    # lists packed; the ids follow the image in the same buffer
    n, s, d = _graphs(40, 3000, 20000, 20)
    full = gcn.subgraph_build(n, s, d)
    rp, cl = _oracle_csr(n, s, d)
    jobs = [(10, 400, 1000 + i, 10 ** 6) for i in range(6)] + [(5, 300, 7, 100)]
    pipe = gcn.Pipeline(theta=2, max_rounds=3, max_aux=200, seg_len=16, workers=workers,
                        depth=3, pinned=False)
    try:
        ids = [pipe.submit_sample(full, *j) for j in jobs]
        assert ids == list(range(len(jobs)))
        for i, (m, budget, seed, ms) in enumerate(jobs):
            jid, ptr, nb, info = pipe.next()
            assert jid == i
            want_v, want_steps = _oracle_sample(rp, cl, m, budget, seed, ms)
            assert info.steps == want_steps and info.n == want_v.size
            assert info.vertices_offset % 256 == 0
            assert info.vertices_offset >= info.image_bytes
            assert nb == info.vertices_offset + 4 * want_v.size
            buf = _image(ptr, nb)
            got_v = buf[info.vertices_offset:].view(np.int32)
            assert np.array_equal(got_v, want_v)
            # the image equals packing the oracle-checked induced subgraph's
            # reduction directly
            orp, ocl = osample.induce(rp, cl, want_v)
            assert info.nnz_direct == orp[-1]
            red = ored.reduce(orp, ocl, theta=2, max_rounds=3, max_aux=200)
            assert info.naux == len(red["pairs"]) and info.nnz == red["rowptr"][-1]
            direct = gcn.redundancy_reduce(gcn.subgraph_induce(full, want_v), theta=2,
                                           max_rounds=3, max_aux=200)
            ib = gcn.image_bytes(direct, 16)
            assert ib == info.image_bytes
            ref = np.zeros(ib, np.uint8)
            gcn.pack(direct, ref.ctypes.data, ib, 16)
            assert np.array_equal(buf[:ib], ref)
            assert info.sample_ms >= 0.0 and info.build_ms >= 0.0
            pipe.release(jid)
    finally:
        pipe.close()


def test_pipeline_sampled_rejects():
    full = gcn.subgraph_build(10, [0, 1], [1, 2])
    pipe = gcn.Pipeline(workers=1, depth=1, pinned=False)
    try:
        with pytest.raises(gcn.GcnError):
            pipe.submit_sample(full, 3, 2, 0, 10)       # m > budget
        with pytest.raises(gcn.GcnError):
            pipe.submit_sample(full, 1, 11, 0, 10)      # budget > n
    finally:
        pipe.close()


def test_sample_full_size():
    # the benchmarked shape: the 716,847-vertex full graph, 1,000 walkers,
    # 8,000 vertices, the first two minibatch seeds; and the induced
    # subgraph of the first against the oracle's
    wl = synth.SAMPLED["yelpfull"]
    fi = synth.make_full_inputs(wl)
    full = gcn.subgraph_build(wl.n_full, fi.src, fi.dst)
    rp, cl = ograph.subgraph_build(wl.n_full, fi.src, fi.dst)
    grp, gcl = full.csr()
    assert np.array_equal(grp, rp) and np.array_equal(gcl, cl)
    rpl, cll = rp.tolist(), cl.tolist()
    for i in range(2):
        seed = wl.sample_seed(i)
        want, want_steps = _oracle_sample(rpl, cll, wl.m, wl.budget, seed, wl.max_steps)
        got, steps = gcn.sample_frontier(full, wl.m, wl.budget, seed, wl.max_steps)
        assert steps == want_steps and np.array_equal(got, want) and got.size == wl.budget
        if i == 0:
            orp, ocl = osample.induce(rp, cl, want)
            srp, scl = gcn.subgraph_induce(full, got).csr()
            assert np.array_equal(srp, orp) and np.array_equal(scl, ocl)


def test_pipeline_keeps_sampled_graph_alive():
    # the caller may drop its handle right after submitting
    import gc
    n, s, d = _graphs(50, 500, 3000)
    rp, cl = _oracle_csr(n, s, d)
    pipe = gcn.Pipeline(theta=2, max_rounds=2, workers=2, depth=2, pinned=False)
    try:
        pipe.submit_sample(gcn.subgraph_build(n, s, d), 4, 100, 77, 10 ** 6)
        gc.collect()
        jid, ptr, nb, info = pipe.next()
        want, _ = _oracle_sample(rp, cl, 4, 100, 77, 10 ** 6)
        got = _image(ptr, nb)[info.vertices_offset:].view(np.int32)
        assert np.array_equal(got, want)
        pipe.release(jid)
    finally:
        pipe.close()


def test_gather_rows_rejects_before_launch():
    # argument checks run before any device call, so they hold without a GPU
    f = gcn._gather_rows
    fake = gcn._vp(4096)
    assert f(None, 16, 10, fake, 5, 16, fake, 16, None) == gcn.E_INVALID_ARG    # NULL src
    assert f(fake, 16, 10, fake, 5, 32, fake, 64, None) == gcn.E_INVALID_ARG    # row > ld_src
    assert f(fake, 64, 10, fake, 5, 32, fake, 16, None) == gcn.E_INVALID_ARG    # row > ld_dst
    assert f(fake, 16, 10, fake, -1, 16, fake, 16, None) == gcn.E_INVALID_ARG   # negative n
    assert f(None, 16, 10, None, 0, 16, None, 16, None) == gcn.OK               # nothing to do
