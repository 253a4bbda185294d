"""Pins of the oracle's GCN step: finite differences, closed forms, planted
mistakes (all on the CPU, float64)."""
import math

import numpy as np
import pytest

from oracle import gcn as og
from oracle import graph as gr
from paper_2001_02498_amd import synth


def _tiny(L, loss, bias, seed):
    """n=12 graph, f_in=5, h=3, C=4; resampled until no pre-activation sits
    within 1e-3 of the ReLU kink."""
    rng = np.random.default_rng(seed)
    for attempt in range(200):
        n = 12
        s, d = synth.random_edges(n, 26, rng)
        rp, cl = gr.subgraph_build(n, s, d)
        X = rng.standard_normal((n, 5))
        params = dict(W_self=[], W_neigh=[], b=[])
        F = 5
        for l in range(L):
            params["W_self"].append(rng.standard_normal((F, 3)) * 0.7)
            params["W_neigh"].append(rng.standard_normal((F, 3)) * 0.7)
            params["b"].append(rng.standard_normal(6) * 0.3 if bias else None)
            F = 6
        params["W_cls"] = rng.standard_normal((6, 4)) * 0.7
        params["b_cls"] = rng.standard_normal(4) * 0.3 if bias else None
        if loss == og.SOFTMAX_CE:
            y = rng.integers(0, 4, size=n)
        else:
            y = (rng.random((n, 4)) < 0.3).astype(np.uint8)
        fw = og.forward(rp, cl, X, params)
        if min(np.abs(z).min() for z in fw["Z"]) > 1e-3:
            return rp, cl, X, params, y
    raise RuntimeError("no kink-free sample")


def _entries(params):
    out = []
    for key in ("W_self", "W_neigh", "b"):
        for l, M in enumerate(params[key]):
            if M is not None:
                out.append((key, l))
    out.append(("W_cls", None))
    if params.get("b_cls") is not None:
        out.append(("b_cls", None))
    return out


def _get(params, key, l):
    return params[key] if l is None else params[key][l]


def _grad_of(grads, key, l):
    name = {"W_self": "dW_self", "W_neigh": "dW_neigh", "b": "db",
            "W_cls": "dW_cls", "b_cls": "db_cls"}[key]
    return grads[name] if l is None else grads[name][l]


def fd_check(rp, cl, X, params, y, loss, eps=1e-6):
    """Largest relative mismatch between analytic and central-difference
    gradients over every weight entry."""
    fw = og.forward(rp, cl, X, params)
    _, dz = og.loss_and_grad(loss, fw["logits"], y)
    grads = og.backward(rp, cl, params, fw, dz)
    worst = 0.0
    for key, l in _entries(params):
        P = _get(params, key, l)
        G = _grad_of(grads, key, l)
        num = np.zeros_like(P)
        for idx in np.ndindex(P.shape):
            old = P[idx]
            P[idx] = old + eps
            lp = og.loss_only(rp, cl, X, params, y, loss)
            P[idx] = old - eps
            lm = og.loss_only(rp, cl, X, params, y, loss)
            P[idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        scale = max(np.abs(num).max(), 1e-12)
        worst = max(worst, np.abs(num - G).max() / scale)
    return worst


@pytest.mark.parametrize("L", [2, 3])
@pytest.mark.parametrize("loss", [og.SOFTMAX_CE, og.SIGMOID_BCE])
@pytest.mark.parametrize("bias", [False, True])
def test_gradients_match_finite_differences(L, loss, bias):
    rp, cl, X, params, y = _tiny(L, loss, bias, seed=100 * L + 10 * loss + bias)
    assert fd_check(rp, cl, X, params, y, loss) < 1e-6


def test_input_gradient_matches_finite_differences():
    """dL/dH_l of Eq. 2c checked by perturbing the layer's input directly."""
    rp, cl, X, params, y = _tiny(3, og.SOFTMAX_CE, False, seed=7)
    fw = og.forward(rp, cl, X, params)
    _, dz = og.loss_and_grad(og.SOFTMAX_CE, fw["logits"], y)
    grads = og.backward(rp, cl, params, fw, dz)
    # dH[0] is dL/dH_1 (output of layer 1): perturb H_1 and run layers 2..3
    H1 = fw["H"][1].copy()

    def loss_from_h1(H):
        sub = dict(W_self=params["W_self"][1:], W_neigh=params["W_neigh"][1:],
                   b=params["b"][1:], W_cls=params["W_cls"], b_cls=None)
        f2 = og.forward(rp, cl, H, sub)
        return og.softmax_ce(f2["logits"], y)[0]
    eps = 1e-6
    num = np.zeros_like(H1)
    for idx in np.ndindex(H1.shape):
        Hp = H1.copy(); Hp[idx] += eps
        Hm = H1.copy(); Hm[idx] -= eps
        num[idx] = (loss_from_h1(Hp) - loss_from_h1(Hm)) / (2 * eps)
    assert np.abs(num - grads["dH"][0]).max() / np.abs(num).max() < 1e-6


def test_zero_weights_closed_forms():
    """All-zero weights give zero logits: loss ln C (softmax) or ln 2 (BCE),
    dlogits = (1/C - onehot)/n or (1/2 - y)/(nC)."""
    rp, cl, X, params, y = _tiny(2, og.SOFTMAX_CE, False, seed=3)
    for key in ("W_self", "W_neigh"):
        params[key] = [np.zeros_like(w) for w in params[key]]
    params["W_cls"] = np.zeros_like(params["W_cls"])
    fw = og.forward(rp, cl, X, params)
    n, C = fw["logits"].shape
    loss, dz = og.softmax_ce(fw["logits"], y)
    assert loss == pytest.approx(math.log(C), rel=1e-15)
    want = np.full((n, C), 1.0 / C)
    want[np.arange(n), y] -= 1.0
    np.testing.assert_allclose(dz, want / n, rtol=1e-15, atol=1e-18)
    yb = (np.arange(n * C).reshape(n, C) % 3 == 0).astype(np.uint8)
    loss, dz = og.sigmoid_bce(fw["logits"], yb)
    assert loss == pytest.approx(math.log(2.0), rel=1e-15)
    np.testing.assert_allclose(dz, (0.5 - yb) / (n * C), rtol=1e-15)


def test_softmax_ce_known_value():
    # two classes, logits (0, ln 3): p = (1/4, 3/4); label 1 -> loss ln(4/3)
    z = np.array([[0.0, math.log(3.0)]])
    loss, dz = og.softmax_ce(z, np.array([1]))
    assert loss == pytest.approx(math.log(4.0 / 3.0), rel=1e-14)
    np.testing.assert_allclose(dz, [[0.25, -0.25]], rtol=1e-14)


def test_bce_known_value_and_stability():
    z = np.array([[0.0, 800.0, -800.0]])
    y = np.array([[1, 1, 0]], dtype=np.uint8)
    loss, dz = og.sigmoid_bce(z, y)
    assert loss == pytest.approx(math.log(2.0) / 3.0, rel=1e-14)
    assert np.all(np.isfinite(dz))


def test_sgd_is_textbook():
    rp, cl, X, params, y = _tiny(2, og.SIGMOID_BCE, True, seed=9)
    out = og.train_step(rp, cl, X, params, y, og.SIGMOID_BCE, 0.25)
    g = out["grads"]
    np.testing.assert_array_equal(out["params"]["W_cls"], params["W_cls"] - 0.25 * g["dW_cls"])
    np.testing.assert_array_equal(out["params"]["W_self"][1],
                                  params["W_self"][1] - 0.25 * g["dW_self"][1])
    np.testing.assert_array_equal(out["params"]["b"][0], params["b"][0] - 0.25 * g["db"][0])


# ------------------------------------------------------------ planted mistakes
# Each plants one plausible mistake into the oracle and checks that a pin
# above catches it; the oracle is restored afterwards by monkeypatch.

def test_planted_transposed_aggregation_is_caught(monkeypatch):
    # backward aggregating with D^-1 A instead of A D^-1
    monkeypatch.setattr(og, "aggregate_transposed",
                        lambda rp, cl, G: og.aggregate(rp, cl, G))
    rp, cl, X, params, y = _tiny(2, og.SOFTMAX_CE, False, seed=22)
    assert fd_check(rp, cl, X, params, y, og.SOFTMAX_CE) > 1e-3


def test_planted_unnormalised_aggregation_is_caught(monkeypatch, golden):
    # forgetting the D^-1 scale breaks the Fig. 1 values
    real = og.aggregate

    def bad(rp, cl, H):
        return og.adjacency(rp, cl, len(rp) - 1) @ np.asarray(H, float)
    monkeypatch.setattr(og, "aggregate", bad)
    g = golden("fig1_aggregation.json")
    e = np.array(g["edges"])
    rp, cl = gr.subgraph_build(g["n"], e[:, 0], e[:, 1])
    assert not np.array_equal(og.aggregate(rp, cl, np.array(g["X"], float)),
                              np.array(g["aggregated"], float))
    monkeypatch.setattr(og, "aggregate", real)


def test_planted_wrong_softmax_sign_is_caught(monkeypatch):
    real = og.softmax_ce

    def bad(z, y):
        loss, dz = real(z, y)
        return loss, -dz
    monkeypatch.setattr(og, "softmax_ce", bad)
    rp, cl, X, params, y = _tiny(2, og.SOFTMAX_CE, False, seed=23)
    assert fd_check(rp, cl, X, params, y, og.SOFTMAX_CE) > 1e-3


def test_planted_missing_mask_is_caught(monkeypatch):
    real_backward = og.backward

    def bad_backward(rp, cl, params, fw, dz):
        fw2 = dict(fw)
        fw2["Z"] = [np.abs(z) + 1.0 for z in fw["Z"]]   # mask always 1
        return real_backward(rp, cl, params, fw2, dz)
    monkeypatch.setattr(og, "backward", bad_backward)
    rp, cl, X, params, y = _tiny(2, og.SOFTMAX_CE, False, seed=24)
    assert fd_check(rp, cl, X, params, y, og.SOFTMAX_CE) > 1e-3


def test_planted_swapped_branches_is_caught(monkeypatch):
    real_forward = og.forward

    def bad_forward(rp, cl, X, params):
        p2 = dict(params)
        p2["W_self"], p2["W_neigh"] = params["W_neigh"], params["W_self"]
        return real_forward(rp, cl, X, p2)
    monkeypatch.setattr(og, "forward", bad_forward)
    rp, cl, X, params, y = _tiny(2, og.SOFTMAX_CE, False, seed=25)
    assert fd_check(rp, cl, X, params, y, og.SOFTMAX_CE) > 1e-3
