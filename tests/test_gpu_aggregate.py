"""GPU parity of the aggregation (pair sums + list sums + degree scaling)
against the oracle's D^-1 A X and A D^-1 X."""
import numpy as np
import pytest

from oracle import gcn as og
from paper_2001_02498_amd import synth
from tests.gpu_helpers import (AGG_TOL, GraphCase, dev, empty, need_gpu, padding_of,
                               rel, say, torch)

pytestmark = pytest.mark.gpu


def _run(case, mode, X, ldx=None, ldy=None):
    gcn = case.gcn
    Xd = dev(X, ldx)
    Y = empty(case.n, X.shape[1], ldy)
    ws = gcn.alloc_ws(gcn.scratch_bytes(case.dg, X.shape[1]))
    gcn.aggregate(case.dg, mode, Xd, Y, ws)
    torch.cuda.synchronize()
    return Y


def test_fig1_values_exact(golden):
    need_gpu()
    g = golden("fig1_aggregation.json")
    e = np.array(g["edges"])
    X = np.array(g["X"], dtype=np.float32)
    for theta, rounds in ((2, 5), (1, 5), (1, 0)):
        say("fig1 theta", theta, "rounds", rounds)
        case = GraphCase(g["n"], e[:, 0], e[:, 1], theta=theta, rounds=rounds)
        Y = _run(case, case.gcn.AGG_MEAN, X)
        assert np.array_equal(Y.cpu().numpy(), np.array(g["aggregated"], np.float32))


@pytest.mark.parametrize("F", [1, 3, 50, 64, 128, 300, 602, 1024, 1100])
@pytest.mark.parametrize("seg_len", [0, 3])
def test_aggregate_widths(F, seg_len):
    need_gpu()
    wl = synth.small_workload(700, 12, 2, 4, 4, 2, synth.SOFTMAX_CE, (F, seg_len))
    inp = synth.make_inputs(wl)
    rng = np.random.default_rng(F)
    X = rng.standard_normal((wl.n, F)).astype(np.float32)
    for rounds in (0, 5):
        say("aggregate F", F, "seg_len", seg_len, "rounds", rounds)
        case = GraphCase(wl.n, inp.src, inp.dst, rounds=rounds, seg_len=seg_len)
        if rounds:
            assert case.info["naux"] > 0
        Y = _run(case, case.gcn.AGG_MEAN, X, ldy=(F + 3) // 4 * 4 + 8)
        assert rel(Y, og.aggregate(case.rp, case.cl, X)) < AGG_TOL
        assert torch.isnan(padding_of(Y)).all()   # padding never written
        Y = _run(case, case.gcn.AGG_TRANSPOSED, X)
        assert rel(Y, og.aggregate_transposed(case.rp, case.cl, X)) < AGG_TOL


@pytest.mark.parametrize("F", [1, 5, 64, 256, 300, 602, 1024, 2100])
def test_aggregate_hubs(F):
    """Hubs (lists of more than 16 pieces): a star on 6,000 vertices, three
    smaller hubs and a sparse background; their workgroups split the
    columns and add the list in a tree, in a fixed order."""
    need_gpu()
    rng = np.random.default_rng(F + 7)
    n = 6000
    src = [np.zeros(n - 1, np.int64)]
    dst = [np.arange(1, n)]
    for h, deg in ((1, 600), (2, 1500), (3, 3100)):
        src.append(np.full(deg, h))
        dst.append(rng.choice(np.arange(4, n), deg, replace=False))
    src.append(rng.integers(4, n, 9000))
    dst.append(rng.integers(4, n, 9000))
    src, dst = np.concatenate(src), np.concatenate(dst)
    X = rng.standard_normal((n, F)).astype(np.float32)
    for rounds, seg_len in ((0, 0), (0, 7), (5, 0)):
        say("hubs F", F, "rounds", rounds, "seg_len", seg_len)
        case = GraphCase(n, src, dst, rounds=rounds, seg_len=seg_len)
        assert case.dg.desc.nhub >= 2
        Y = _run(case, case.gcn.AGG_MEAN, X, ldy=(F + 3) // 4 * 4 + 4)
        assert rel(Y, og.aggregate(case.rp, case.cl, X)) < AGG_TOL
        assert torch.isnan(padding_of(Y)).all()
        Y2 = _run(case, case.gcn.AGG_MEAN, X, ldy=(F + 3) // 4 * 4 + 4)
        assert torch.equal(Y, Y2)
        Y = _run(case, case.gcn.AGG_TRANSPOSED, X)
        assert rel(Y, og.aggregate_transposed(case.rp, case.cl, X)) < AGG_TOL


def test_aggregate_integer_features_direct_equals_reduced():
    """Integer features: every partial sum is exact in fp32, so the reduced
    graph reaches D^-1 A X bit for bit (same rounding of the final scale)."""
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    inp = synth.make_inputs(wl)
    rng = np.random.default_rng(0)
    X = rng.integers(-8, 9, size=(wl.n, 64)).astype(np.float32)
    direct = GraphCase(wl.n, inp.src, inp.dst, rounds=0)
    red = GraphCase(wl.n, inp.src, inp.dst, rounds=5)
    a = _run(direct, direct.gcn.AGG_MEAN, X).cpu().numpy()
    b = _run(red, red.gcn.AGG_MEAN, X).cpu().numpy()
    assert np.array_equal(a, b)


def test_aggregate_workload_ppi_reduced_and_direct():
    need_gpu()
    wl = synth.WORKLOADS["ppi8k"]
    inp = synth.make_inputs(wl)
    rng = np.random.default_rng(1)
    for F in (50, 1024):
        X = rng.standard_normal((wl.n, F)).astype(np.float32)
        ref = og.aggregate(*synth_csr(wl, inp), X)
        for rounds in (0, wl.rounds):
            say("ppi8k F", F, "rounds", rounds)
            case = GraphCase(wl.n, inp.src, inp.dst, theta=wl.theta, rounds=rounds,
                             max_aux=wl.max_aux)
            Y = _run(case, case.gcn.AGG_MEAN, X)
            assert rel(Y, ref) < AGG_TOL


def test_aggregate_isolated_and_empty():
    need_gpu()
    # vertices 3 and 4 isolated; a graph with no edges at all
    case = GraphCase(5, np.array([0, 1]), np.array([1, 2]))
    X = np.arange(5 * 6, dtype=np.float32).reshape(5, 6)
    Y = _run(case, case.gcn.AGG_MEAN, X).cpu().numpy()
    assert np.all(Y[3:] == 0)
    case = GraphCase(4, np.zeros(0, np.int64), np.zeros(0, np.int64))
    Y = _run(case, case.gcn.AGG_TRANSPOSED, X[:4]).cpu().numpy()
    assert np.all(Y == 0)


def test_aggregate_deterministic():
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    inp = synth.make_inputs(wl)
    case = GraphCase(wl.n, inp.src, inp.dst, seg_len=5)
    X = np.random.default_rng(2).standard_normal((wl.n, 256)).astype(np.float32)
    a = _run(case, case.gcn.AGG_MEAN, X).cpu()
    b = _run(case, case.gcn.AGG_MEAN, X).cpu()
    assert torch.equal(a, b)


def synth_csr(wl, inp):
    from oracle import graph as gr
    return gr.subgraph_build(wl.n, inp.src, inp.dst)
