"""The device redundancy reduction (gcn_redundancy_reduce_device) equals the
oracle's Algorithms 1-3 field by field -- pairs, round offsets, rewritten
lists and per-round counts -- on every case here, and the host reduction as
well."""
import numpy as np
import pytest

from oracle import graph as gr
from oracle import reduction as rd
from paper_2001_02498_amd import synth
from tests.gpu_helpers import need_gpu, say

pytestmark = pytest.mark.gpu


def _both(gcn, n, s, d, **kw):
    """Device and host reductions, the device one also checked against the
    oracle's reduction of the oracle's own subgraph."""
    g = gcn.subgraph_build(n, s, d)
    host = gcn.redundancy_reduce(g, **kw).info()
    ws = gcn.alloc_ws(max(gcn.redundancy_reduce_device_bytes(g, **kw), 256))
    dev = gcn.redundancy_reduce_device(g, ws, **kw).info()
    rp, cl = gr.subgraph_build(n, s, d)
    _same_as_oracle(dev, rd.reduce(rp, cl, **kw))
    return host, dev


def _same_as_oracle(dev, ora):
    assert dev["naux"] == ora["naux"]
    assert np.array_equal(dev["pairs"], np.asarray(ora["pairs"], np.int32).reshape(-1, 2))
    for k in ("round_offsets", "rowptr", "col"):
        assert np.array_equal(dev[k], ora[k]), k
    assert [tuple(x) for x in dev["stats"]] == [tuple(x) for x in ora["stats"]]


def _same(host, dev):
    for k in ("naux", "rounds"):
        assert host[k] == dev[k], k
    for k in ("pairs", "round_offsets", "rowptr", "col", "deg"):
        assert np.array_equal(host[k], dev[k]), k
    assert [tuple(x) for x in host["stats"]] == [tuple(x) for x in dev["stats"]]


def test_device_reduction_random_graphs():
    need_gpu()
    from paper_2001_02498_amd import gcn
    rng = np.random.default_rng(31)
    for trial in range(40):
        n = int(rng.integers(2, 400))
        s, d = synth.random_edges(n, int(rng.integers(0, 12 * n)), rng)
        kw = dict(theta=int(rng.integers(0, 4)), max_rounds=int(rng.integers(0, 7)),
                  max_aux=int(rng.integers(-1, 3 * n // 4)))
        say("device reduction", trial, n, len(s), kw)
        host, dev = _both(gcn, n, s, d, **kw)
        _same(host, dev)


def test_device_reduction_figures(golden):
    need_gpu()
    from paper_2001_02498_amd import gcn
    g1 = golden("fig1_aggregation.json")
    e = np.array(g1["edges"])
    g = gcn.subgraph_build(g1["n"], e[:, 0], e[:, 1])
    ws = gcn.alloc_ws(gcn.redundancy_reduce_device_bytes(g, theta=1))
    info = gcn.redundancy_reduce_device(g, ws, theta=1).info()
    want = golden("fig1_reduction.json")
    assert info["pairs"].tolist() == want["pairs"]
    assert info["rowptr"].tolist() == want["rowptr"]
    assert info["col"].tolist() == want["col"]
    rp, cl = gr.subgraph_build(g1["n"], e[:, 0], e[:, 1])
    ora = rd.reduce(rp, cl, theta=1)
    assert np.array_equal(info["col"], ora["col"])


@pytest.mark.parametrize("name", ["tiny", "ppi8k", "yelp10k", "reddit8k", "stream8k"])
def test_device_reduction_workloads(name):
    need_gpu()
    from paper_2001_02498_amd import gcn
    wl = synth.WORKLOADS[name]
    inp = synth.make_inputs(wl)
    say("device reduction", name)
    host, dev = _both(gcn, wl.n, inp.src, inp.dst, theta=wl.theta, max_rounds=5,
                      max_aux=wl.max_aux)
    _same(host, dev)
    assert dev["naux"] > 0


def test_device_reduction_stream_subgraphs():
    need_gpu()
    from paper_2001_02498_amd import gcn
    for i in (1, 7, 63):
        wl = synth.stream_workload(i)
        inp = synth.make_inputs(wl)
        host, dev = _both(gcn, wl.n, inp.src, inp.dst, theta=wl.theta, max_rounds=wl.rounds,
                          max_aux=wl.max_aux)
        _same(host, dev)


def test_device_reduction_edges_and_errors():
    need_gpu()
    from paper_2001_02498_amd import gcn
    # edgeless and single-edge graphs, zero rounds, zero budget
    for (n, s, d) in [(5, [], []), (2, [0], [1]), (1, [], [])]:
        for kw in (dict(), dict(max_rounds=0), dict(max_aux=0), dict(theta=0)):
            host, dev = _both(gcn, n, np.array(s, np.int64), np.array(d, np.int64), **kw)
            _same(host, dev)
    g = gcn.subgraph_build(50, *synth.random_edges(50, 300, np.random.default_rng(2)))
    need = gcn.redundancy_reduce_device_bytes(g)
    with pytest.raises(gcn.GcnError) as ei:
        gcn.redundancy_reduce_device(g, gcn.alloc_ws(need // 2 // 256 * 256 or 256))
    assert ei.value.code == gcn.E_WORKSPACE


def test_device_reduction_beyond_16bit_ids():
    """More ids than 16-bit counters cover: Algorithm 1 counts in windows of
    65,536 ids (from the first round at n = 70,000, with the 16-bit counter
    overflow check on; from the second round at n = 65,400, whose first
    round's pair sums push the ids past 65,536)."""
    need_gpu()
    from paper_2001_02498_amd import gcn
    for n, oracle in ((70000, True), (65400, False)):
        wl = synth.small_workload(n, 4, 2, 8, 8, 4, synth.SOFTMAX_CE, (n,))
        inp = synth.make_inputs(wl)
        kw = dict(theta=2, max_rounds=5)
        say("device reduction", n, len(inp.src), "oracle", oracle)
        if oracle:
            host, dev = _both(gcn, n, inp.src, inp.dst, **kw)
        else:
            g = gcn.subgraph_build(n, inp.src, inp.dst)
            host = gcn.redundancy_reduce(g, **kw).info()
            ws = gcn.alloc_ws(gcn.redundancy_reduce_device_bytes(g, **kw))
            dev = gcn.redundancy_reduce_device(g, ws, **kw).info()
        _same(host, dev)
        assert n + dev["round_offsets"][1] > 65536 and dev["rounds"] >= 2

