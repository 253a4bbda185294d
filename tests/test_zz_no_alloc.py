"""gcn_aggregate_noalloc (the aggregation on the library's fixed per-device
scratch, for callers that cannot allocate) against gcn_aggregate with a
caller workspace: identical results, call after call, with the second call
on a smaller input, and a clear error beyond the fixed scratch size."""
import numpy as np
import pytest

from oracle import gcn as og
from paper_2001_02498_amd import synth
from tests.gpu_helpers import AGG_TOL, GraphCase, dev, empty, need_gpu, rel, say, torch

pytestmark = pytest.mark.gpu


def _case(name):
    wl = synth.WORKLOADS[name]
    inp = synth.make_inputs(wl)
    return GraphCase(wl.n, inp.src, inp.dst, theta=wl.theta, rounds=wl.rounds,
                     max_aux=wl.max_aux)


def _both(gcn, case, mode, F, seed):
    rng = np.random.default_rng(seed)
    X = dev(rng.standard_normal((case.n, F)).astype(np.float32))
    need = gcn.scratch_bytes(case.dg, F)
    ws = gcn.alloc_ws(need)
    Y_ws = empty(case.n, F)
    gcn.aggregate(case.dg, mode, X, Y_ws, ws)
    Y_na = empty(case.n, F)
    say("aggregate_noalloc", case.n, "naux", case.info["naux"], "F", F, "mode", mode)
    gcn.aggregate_noalloc(case.dg, mode, X, Y_na)
    torch.cuda.synchronize()
    return X, Y_ws, Y_na


def test_noalloc_equals_workspace_entry_point():
    need_gpu()
    from paper_2001_02498_amd import gcn
    big, small = _case("ppi8k"), _case("tiny")
    # a large call, then a smaller one (smaller graph and width) on the same
    # device array, then the large one again in the transposed mode
    for case, mode, F, seed in ((big, gcn.AGG_MEAN, 1024, 1), (small, gcn.AGG_MEAN, 64, 2),
                                (big, gcn.AGG_TRANSPOSED, 512, 3), (small, gcn.AGG_TRANSPOSED, 37, 4)):
        X, Y_ws, Y_na = _both(gcn, case, mode, F, seed)
        assert torch.equal(Y_ws, Y_na), (case.n, mode, F)
        # and the oracle's definition (D^-1 A X, or A D^-1 X)
        Xn = X.cpu().double().numpy()
        f = og.aggregate if mode == gcn.AGG_MEAN else og.aggregate_transposed
        assert rel(Y_na, f(case.rp, case.cl, Xn)) < AGG_TOL


def test_noalloc_rejects_beyond_fixed_scratch():
    need_gpu()
    from paper_2001_02498_amd import gcn
    case = _case("ppi8k")
    F = 8192   # 4 F naux alone is 86 MB > 64 MiB
    assert 4 * F * case.info["naux"] > gcn.AGG_NOALLOC_SCRATCH_BYTES
    X = dev(np.ones((case.n, F), np.float32))
    Y = empty(case.n, F)
    with pytest.raises(gcn.GcnError) as e:
        gcn.aggregate_noalloc(case.dg, gcn.AGG_MEAN, X, Y)
    assert e.value.code == gcn.E_INVALID_ARG
    assert "exceed the fixed" in str(e.value)
    torch.cuda.synchronize()
    assert torch.isnan(Y).all()   # nothing launched
