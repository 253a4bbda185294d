"""GPU parity of the layer-level entry points (forward transform, classifier,
loss, backward with fused update) against the oracle, at sizes spanning
several 128 x 128 tiles with ragged edges."""
import math

import numpy as np
import pytest

from oracle import gcn as og
from paper_2001_02498_amd import synth
from tests.gpu_helpers import (FP32_TOL, GraphCase, dev, empty, need_gpu, padding_of, rel,
                               say, torch)

pytestmark = pytest.mark.gpu


def _graph(n, seed, rounds=5, seg_len=0):
    wl = synth.small_workload(n, 14, 2, 4, 4, 2, synth.SOFTMAX_CE, (seed,))
    inp = synth.make_inputs(wl)
    return GraphCase(n, inp.src, inp.dst, rounds=rounds, seg_len=seg_len)


def _ws(case, W):
    return case.gcn.alloc_ws(case.gcn.scratch_bytes(case.dg, W))


# (9000, 64, 256): a 40-row last row tile, two products of 256 columns
@pytest.mark.parametrize("n,F,h,bias", [(777, 50, 36, False), (1024, 64, 128, True),
                                        (300, 602, 20, False), (513, 256, 132, True),
                                        (9000, 64, 256, True)])
def test_layer_fwd(n, F, h, bias):
    need_gpu()
    say("layer_fwd", n, F, h, bias)
    case = _graph(n, F)
    gcn = case.gcn
    rng = np.random.default_rng(F + h)
    X = rng.standard_normal((n, F)).astype(np.float32)
    Ws = synth.glorot(rng, F, h)
    Wn = synth.glorot(rng, F, h)
    b = (rng.standard_normal(2 * h) * 0.1).astype(np.float32) if bias else None
    AH = empty(n, F)
    H = empty(n, 2 * h, (2 * h + 3) // 4 * 4 + 4)
    gcn.layer_fwd(case.dg, dev(X), dev(Ws, h), dev(Wn, h), dev(b) if bias else None,
                  AH, H, _ws(case, max(F, 2 * h)))
    torch.cuda.synchronize()
    AH_ref = og.aggregate(case.rp, case.cl, X)
    Z = np.concatenate([X.astype(float) @ Ws, AH_ref @ Wn], axis=1)
    if bias:
        Z = Z + b
    assert rel(AH, AH_ref) < 1e-5
    assert rel(H, np.maximum(Z, 0)) < FP32_TOL
    assert torch.isnan(padding_of(H)).all()


# (the weight gradient runs on 32 x 128 tiles: the cases cover a ragged
# last row tile holding the bias row, two column tiles and a short M; the
# logits on 64 x 128 tiles, with K slices below 256 row tiles and without
# them at n = 17000)
@pytest.mark.parametrize("n,K,C,bias", [(1000, 256, 121, True), (333, 64, 16, False),
                                        (129, 1024, 41, False), (700, 96, 200, True),
                                        (2000, 36, 7, True), (17000, 64, 10, True)])
def test_classifier_fwd_loss_bwd(n, K, C, bias):
    need_gpu()
    say("classifier", n, K, C, bias)
    from paper_2001_02498_amd import gcn
    rng = np.random.default_rng(n + K + C)
    H = np.maximum(rng.standard_normal((n, K)), 0).astype(np.float32)
    Wc = synth.glorot(rng, K, C)
    bc = (rng.standard_normal(C) * 0.1).astype(np.float32) if bias else None
    Hd, Wd = dev(H), torch.from_numpy(Wc.copy()).cuda()
    bd = torch.from_numpy(bc.copy()).cuda() if bias else None
    Z = empty(n, C)
    ws = gcn.alloc_ws(gcn.scratch_bytes(None, max(K, C), n=n))
    gcn.classifier_fwd(Hd, K, Wd, bd, Z, ws)
    Zref = H.astype(float) @ Wc + (bc if bias else 0)
    torch.cuda.synchronize()
    assert rel(Z, Zref) < FP32_TOL
    assert torch.isnan(padding_of(Z)).all()
    for kind in (og.SOFTMAX_CE, og.SIGMOID_BCE):
        if kind == og.SOFTMAX_CE:
            y = rng.integers(0, C, n).astype(np.int32)
        else:
            y = (rng.random((n, C)) < 0.2).astype(np.uint8)
        yd = torch.from_numpy(y).cuda()
        dZ = empty(n, C)
        loss = torch.zeros(1, device="cuda")
        gcn.loss(kind, Z, C, yd, dZ, loss, ws)
        torch.cuda.synchronize()
        Zg = Z.cpu().double().numpy()        # the loss is checked on the same logits
        lref, dref = og.loss_and_grad(kind, Zg, y)
        assert abs(loss.item() - lref) <= 1e-5 * abs(lref)
        assert rel(dZ, dref) < 1e-5
        # backward: G = (dZ W^T) * [H > 0]; dW = H^T dZ; W -= lr dW
        W2 = Wd.clone()
        b2 = bd.clone() if bias else None
        G = empty(n, K)
        dW = torch.zeros_like(Wd)
        db = torch.zeros(C, device="cuda") if bias else None
        lr = 0.5
        gcn.classifier_bwd(dZ, C, Hd, K, W2, b2, lr, G, dW, db, ws)
        torch.cuda.synchronize()
        dZh = dZ.cpu().double().numpy()
        Gref = (dZh @ Wc.T.astype(float)) * (H > 0)
        dWref = H.T.astype(float) @ dZh
        assert rel(G, Gref) < FP32_TOL
        assert rel(dW, dWref) < FP32_TOL
        new = W2.cpu().double().numpy()
        assert rel(new - Wc, -lr * dWref) < FP32_TOL
        if bias:
            assert rel(db, dZh.sum(0)) < FP32_TOL
            assert rel(b2.cpu().double().numpy() - bc, -lr * dZh.sum(0)) < FP32_TOL


@pytest.mark.parametrize("n,F,h,bias,first", [(777, 50, 36, False, True),
                                              (1024, 256, 128, True, False),
                                              (300, 602, 20, False, False),
                                              (1500, 1024, 132, True, False),
                                              # weight gradients with at most 64
                                              # rows (both wavefront rows split K)
                                              # and just past that bound
                                              (5000, 64, 128, True, True),
                                              (5000, 63, 72, True, True),
                                              (2000, 65, 40, False, True),
                                              (4100, 8, 24, False, True),
                                              # a 40-row last row tile
                                              (9000, 512, 64, True, False)])
def test_layer_bwd(n, F, h, bias, first):
    need_gpu()
    say("layer_bwd", n, F, h, bias, first)
    case = _graph(n, F + 1, seg_len=16)
    gcn = case.gcn
    rng = np.random.default_rng(F * 3 + h)
    H_in = rng.standard_normal((n, F)).astype(np.float32)
    if not first:
        H_in = np.maximum(H_in, 0)
    AH = og.aggregate(case.rp, case.cl, H_in).astype(np.float32)
    G = (rng.standard_normal((n, 2 * h)) * (rng.random((n, 2 * h)) < 0.6)).astype(np.float32)
    Ws, Wn = synth.glorot(rng, F, h), synth.glorot(rng, F, h)
    b = (rng.standard_normal(2 * h) * 0.1).astype(np.float32) if bias else None
    Wsd, Wnd = dev(Ws, h), dev(Wn, h)
    bd = dev(b) if bias else None
    G_in = None if first else empty(n, F)
    dWs, dWn = torch.zeros_like(Wsd), torch.zeros_like(Wnd)
    db = torch.zeros(2 * h, device="cuda") if bias else None
    lr = 0.25
    gcn.layer_bwd(case.dg, dev(G), dev(H_in), dev(AH), Wsd, Wnd, bd, lr, G_in, dWs, dWn, db,
                  _ws(case, max(F, 2 * h)))
    torch.cuda.synchronize()
    Gs, Gn = G[:, :h].astype(float), G[:, h:].astype(float)
    dWs_ref = H_in.T.astype(float) @ Gs
    dWn_ref = AH.T.astype(float) @ Gn
    assert rel(dWs, dWs_ref) < FP32_TOL
    assert rel(dWn, dWn_ref) < FP32_TOL
    assert rel(Wsd.cpu().double().numpy() - Ws, -lr * dWs_ref) < FP32_TOL
    assert rel(Wnd.cpu().double().numpy() - Wn, -lr * dWn_ref) < FP32_TOL
    if bias:
        assert rel(db, G.astype(float).sum(0)) < FP32_TOL
    if not first:
        ref = (Gs @ Ws.T + og.aggregate_transposed(case.rp, case.cl, Gn) @ Wn.T) * (H_in > 0)
        assert rel(G_in, ref) < FP32_TOL
        assert torch.isnan(padding_of(G_in)).all()


def test_layer_errors_before_launch():
    need_gpu()
    case = _graph(100, 1)
    gcn = case.gcn
    X = dev(np.zeros((100, 8), np.float32))
    AH, H = empty(100, 8), empty(100, 16)
    W = dev(np.zeros((8, 8), np.float32), 8)
    with pytest.raises(gcn.GcnError) as ei:       # workspace too small
        gcn.layer_fwd(case.dg, X, W, W, None, AH, H, gcn.alloc_ws(256))
    assert ei.value.code == gcn.E_WORKSPACE
    with pytest.raises(gcn.GcnError) as ei:       # h not a multiple of 4
        W6 = dev(np.zeros((8, 6), np.float32), 8)[:, :6].contiguous()
        gcn.layer_fwd(case.dg, X, W6, W6, None, AH, empty(100, 12), _ws(case, 16))
    assert ei.value.code == gcn.E_INVALID_ARG
    with pytest.raises(gcn.GcnError) as ei:
        gcn.layer_fwd(case.dg, X, W, W, None, AH, H, _ws(case, 16), precision=7)
    assert ei.value.code == gcn.E_INVALID_ARG
    assert torch.isnan(H).all()     # outputs untouched on error
