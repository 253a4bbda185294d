"""The loss status word: invalid labels (a softmax class outside [0, C), a
multi-label byte other than 0 or 1) and a non-finite loss are written on
the device by every loss call and training step, and reported by
gcn_status_check at the next host sync; a later valid call clears them."""
import dataclasses

import numpy as np
import pytest

from paper_2001_02498_amd import synth
from tests.gpu_helpers import dev, empty, need_gpu, say, torch

pytestmark = pytest.mark.gpu


def _loss_call(gcn, kind, Z, labels, C):
    n = Z.shape[0]
    ws = gcn.alloc_ws(gcn.scratch_bytes(None, C, n=n))
    dZ = empty(n, C)
    loss = torch.zeros(1, device="cuda")
    gcn.loss(kind, Z, C, labels, dZ, loss, ws)
    return ws, loss


def _status(gcn, ws, offset=0):
    try:
        gcn.status_check(ws, offset)
        return gcn.OK
    except gcn.GcnError as e:
        return e.code


def test_loss_status_labels_and_nonfinite():
    need_gpu()
    from paper_2001_02498_amd import gcn
    rng = np.random.default_rng(11)
    n, C = 300, 41
    Z = dev(rng.standard_normal((n, C)).astype(np.float32))
    y = rng.integers(0, C, n).astype(np.int32)
    ws, _ = _loss_call(gcn, gcn.LOSS_SOFTMAX_CE, Z, torch.from_numpy(y).cuda(), C)
    assert _status(gcn, ws) == 0
    for bad in (C, -1, 1 << 20):
        yb = y.copy()
        yb[137] = bad
        say("softmax label", bad)
        ws, _ = _loss_call(gcn, gcn.LOSS_SOFTMAX_CE, Z, torch.from_numpy(yb).cuda(), C)
        assert _status(gcn, ws) == gcn.E_INVALID_ARG
        assert "label" in gcn.last_error()
    # multi-label: bytes other than 0 / 1
    Yb = (rng.random((n, C)) < 0.2).astype(np.uint8)
    ws, _ = _loss_call(gcn, gcn.LOSS_SIGMOID_BCE, Z, torch.from_numpy(Yb).cuda(), C)
    assert _status(gcn, ws) == 0
    Yb[5, 40] = 2
    ws, _ = _loss_call(gcn, gcn.LOSS_SIGMOID_BCE, Z, torch.from_numpy(Yb).cuda(), C)
    assert _status(gcn, ws) == gcn.E_INVALID_ARG
    # a non-finite logit makes the loss non-finite
    for kind, lab, bad in ((gcn.LOSS_SOFTMAX_CE, torch.from_numpy(y).cuda(), np.inf),
                           (gcn.LOSS_SIGMOID_BCE,
                            torch.from_numpy((Yb > 0).astype(np.uint8)).cuda(), np.nan)):
        Zh = Z.cpu().numpy().copy()
        Zh[3, 7] = bad
        ws, loss = _loss_call(gcn, kind, dev(Zh), lab, C)
        assert _status(gcn, ws) == gcn.E_NONFINITE
        assert not np.isfinite(loss.item())
        # the same workspace, a valid call: the word is rewritten
        gcn.loss(kind, Z, C, lab, empty(n, C), loss, ws)
        assert _status(gcn, ws) == 0


def test_train_step_status():
    need_gpu()
    from paper_2001_02498_amd import gcn
    from tests.test_gpu_step import StepRun
    wl = synth.WORKLOADS["tiny"]
    inp = synth.make_inputs(wl)
    good = StepRun(wl, inp=inp).run()
    assert _status(gcn, good.ws, good.layout.status) == 0
    bad_labels = inp.labels.copy()
    bad_labels[5] = wl.C
    bad = StepRun(wl, inp=dataclasses.replace(inp, labels=bad_labels)).run()
    assert _status(gcn, bad.ws, bad.layout.status) == gcn.E_INVALID_ARG
    # a NaN or an infinity among the features reaches the loss through the
    # aggregation, the products and the ReLUs (which keep a NaN)
    for bad in (np.nan, np.inf):
        X = inp.X.copy()
        X[0, 0] = bad
        nf = StepRun(wl, inp=dataclasses.replace(inp, X=X)).run()
        assert _status(gcn, nf.ws, nf.layout.status) == gcn.E_NONFINITE, bad
