"""Pins of the oracle's optimiser updates (oracle/optim.py) against what the
mathematics fixes: closed forms under a constant gradient, special cases
that reduce to plain gradient descent, and the structure of the model-wide
update."""
import numpy as np
import pytest

from oracle import gcn as og
from oracle import optim as oo

RNG = np.random.default_rng(11)


def test_momentum_zero_is_gradient_descent():
    W, g = RNG.standard_normal((5, 3)), RNG.standard_normal((5, 3))
    u0 = RNG.standard_normal((5, 3))
    opt = oo.Optim(oo.MOMENTUM, lr=0.1, momentum=0.0)
    W1, u1, _ = oo.update(opt, W, g, u0)
    assert np.array_equal(u1, g)
    assert np.allclose(W1, W - 0.1 * g, rtol=0, atol=1e-15)


@pytest.mark.parametrize("mu", [0.5, 0.9])
def test_momentum_constant_gradient_closed_form(mu):
    # u_t = g (1 - mu^t) / (1 - mu);  W_t = W_0 - lr g sum_k (1 - mu^k) / (1 - mu)
    #     = W_0 - lr g (t - mu (1 - mu^t) / (1 - mu)) / (1 - mu)
    W0, g = RNG.standard_normal(7), RNG.standard_normal(7)
    lr, T = 0.05, 12
    opt = oo.Optim(oo.MOMENTUM, lr=lr, momentum=mu)
    W, u = W0.copy(), np.zeros(7)
    for t in range(1, T + 1):
        W, u, _ = oo.update(opt, W, g, u)
        assert np.allclose(u, g * (1 - mu ** t) / (1 - mu), rtol=1e-13, atol=0)
    closed = W0 - lr * g * (T - mu * (1 - mu ** T) / (1 - mu)) / (1 - mu)
    assert np.allclose(W, closed, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("eps", [1e-8, 0.5])
def test_adam_constant_gradient_closed_form(eps):
    # with g constant, the bias-corrected moments are exactly g and g^2 for
    # every t, so each update is lr g / (|g| + eps) (a large eps tells
    # eps outside the square root from eps inside it)
    W0 = RNG.standard_normal(9)
    g = RNG.standard_normal(9) * np.array([1e-3, 1e-2, 0.1, 1, 10, 100, 1, 1, 1])
    lr, T = 0.01, 6
    opt = oo.Optim(oo.ADAM, lr=lr, beta1=0.9, beta2=0.999, eps=eps)
    W, m, v = W0.copy(), np.zeros(9), np.zeros(9)
    for t in range(1, T + 1):
        opt.step = t
        W, m, v = oo.update(opt, W, g, m, v)
        assert np.allclose(m, g * (1 - 0.9 ** t), rtol=1e-12)
        assert np.allclose(v, g * g * (1 - 0.999 ** t), rtol=1e-12)
    assert np.allclose(W, W0 - T * lr * g / (np.abs(g) + eps), rtol=1e-12, atol=1e-15)


def test_adam_without_averaging_is_normalised_descent():
    # beta1 = beta2 = 0: m = g, v = g^2 whatever the history and the step
    W0 = RNG.standard_normal(6)
    opt = oo.Optim(oo.ADAM, lr=0.2, step=3, beta1=0.0, beta2=0.0, eps=1e-3)
    g = RNG.standard_normal(6)
    W, m, v = oo.update(opt, W0, g, RNG.standard_normal(6), RNG.random(6))
    assert np.array_equal(m, g) and np.array_equal(v, g * g)
    assert np.allclose(W, W0 - 0.2 * g / (np.abs(g) + 1e-3), rtol=1e-14)


def test_adam_first_step_is_sign_step():
    # from zero state the first update is lr g / (|g| + eps): lr sign(g) for |g| >> eps
    W0 = RNG.standard_normal(5)
    g = np.array([3.0, -2.0, 0.5, -1e-2, 7.0])
    opt = oo.Optim(oo.ADAM, lr=0.01, step=1, eps=1e-12)
    W, _, _ = oo.update(opt, W0, g, np.zeros(5), np.zeros(5))
    assert np.allclose(W, W0 - 0.01 * np.sign(g), rtol=0, atol=1e-11)


def test_adam_two_steps_by_hand():
    # g = 1 then 3, beta1 0.9, beta2 0.999, eps 0: after step 2
    #   m = 0.1*0.9*1 + 0.1*3 = 0.39,  m_hat = 0.39 / 0.19
    #   v = 0.001*0.999*1 + 0.001*9 = 0.009999,  v_hat = 0.009999 / 0.001999
    opt = oo.Optim(oo.ADAM, lr=1.0, beta1=0.9, beta2=0.999, eps=0.0)
    W, m, v = np.zeros(1), np.zeros(1), np.zeros(1)
    opt.step = 1
    W1, m, v = oo.update(opt, W, np.array([1.0]), m, v)
    assert np.allclose(W1, -1.0)
    opt.step = 2
    W2, m, v = oo.update(opt, W1, np.array([3.0]), m, v)
    assert np.allclose(m, 0.39) and np.allclose(v, 0.009999)
    step2 = (0.39 / 0.19) / np.sqrt(0.009999 / 0.001999)
    assert np.allclose(W2, -1.0 - step2, rtol=1e-14)
    assert 0.917 < step2 < 0.918


def test_sgd_kind_matches_plain_descent_in_the_step():
    # the oracle step with opt = SGD equals its plain-descent path
    from oracle import graph as gr
    from paper_2001_02498_amd import synth
    wl = synth.small_workload(60, 5, 2, 7, 8, 3, synth.SOFTMAX_CE, (3,))
    inp = synth.make_inputs(wl)
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    params = dict(W_self=inp.W_self, W_neigh=inp.W_neigh, b=[None] * wl.L, W_cls=inp.W_cls,
                  b_cls=None)
    a = og.train_step(rp, cl, inp.X, params, inp.labels, wl.loss, 0.03)
    b = og.train_step(rp, cl, inp.X, params, inp.labels, wl.loss, 0.0,
                      opt=oo.Optim(oo.SGD, lr=0.03))
    for l in range(wl.L):
        assert np.array_equal(a["params"]["W_self"][l], b["params"]["W_self"][l])
        assert np.array_equal(a["params"]["W_neigh"][l], b["params"]["W_neigh"][l])
    assert np.array_equal(a["params"]["W_cls"], b["params"]["W_cls"])


def test_apply_updates_every_weight_and_bias_with_its_own_state():
    L = 2
    shapes = dict(W_self=[(4, 3), (6, 3)], W_neigh=[(4, 3), (6, 3)], b=[(6,), (6,)])
    params = {k: [RNG.standard_normal(s) for s in v] for k, v in shapes.items()}
    params["W_cls"], params["b_cls"] = RNG.standard_normal((6, 2)), RNG.standard_normal(2)
    grads = {"d" + k: [RNG.standard_normal(s) for s in v] for k, v in shapes.items()}
    grads["dW_cls"], grads["db_cls"] = RNG.standard_normal((6, 2)), RNG.standard_normal(2)
    state = {k: [RNG.standard_normal(s) for s in v] for k, v in shapes.items()}
    state["W_cls"], state["b_cls"] = RNG.standard_normal((6, 2)), RNG.standard_normal(2)
    opt = oo.Optim(oo.MOMENTUM, lr=0.1, momentum=0.7)
    new, s1, s2 = oo.apply(opt, params, grads, state)
    assert s2["W_cls"] is None
    for k in shapes:
        for l in range(L):
            u = 0.7 * state[k][l] + grads["d" + k][l]
            assert np.allclose(s1[k][l], u)
            assert np.allclose(new[k][l], params[k][l] - 0.1 * u)
    assert np.allclose(new["b_cls"], params["b_cls"] - 0.1 * (0.7 * state["b_cls"]
                                                              + grads["db_cls"]))
