"""Optimiser updates of the weights for the oracle, float64 throughout.

TEST INFRASTRUCTURE ONLY (see the package header).

Section 4.1 lists what each optimiser keeps beside the weights: nothing for
plain gradient descent, the earlier steps' weight gradients for gradient
descent with momentum, and first and second moment estimates for Adam. The
paper defers the update rules to the cited methods; they are, for one weight
W with this step's gradient g:

  gradient descent:   W <- W - lr g
  momentum (heavy ball, the velocity u accumulates the gradients):
                      u <- mu u + g
                      W <- W - lr u
  Adam, update number t = 1, 2, ...:
                      m <- beta1 m + (1 - beta1) g
                      v <- beta2 v + (1 - beta2) g^2
                      W <- W - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

The states start at zero before the first update.
"""
from __future__ import annotations

import dataclasses

import numpy as np

SGD = 0
MOMENTUM = 1
ADAM = 2


@dataclasses.dataclass
class Optim:
    kind: int = SGD
    lr: float = 0.01
    step: int = 1            # Adam: number of this update, from 1
    momentum: float = 0.9
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


def update(opt: Optim, W, g, s1=None, s2=None):
    """One weight's update; returns (W_new, s1_new, s2_new) (None for state
    the optimiser does not keep)."""
    W = np.asarray(W, np.float64)
    g = np.asarray(g, np.float64)
    if opt.kind == SGD:
        return W - opt.lr * g, None, None
    if opt.kind == MOMENTUM:
        u = opt.momentum * np.asarray(s1, np.float64) + g
        return W - opt.lr * u, u, None
    if opt.kind == ADAM:
        m = opt.beta1 * np.asarray(s1, np.float64) + (1.0 - opt.beta1) * g
        v = opt.beta2 * np.asarray(s2, np.float64) + (1.0 - opt.beta2) * g * g
        m_hat = m / (1.0 - opt.beta1 ** opt.step)
        v_hat = v / (1.0 - opt.beta2 ** opt.step)
        return W - opt.lr * m_hat / (np.sqrt(v_hat) + opt.eps), m, v
    raise ValueError(f"unknown optimiser kind {opt.kind}")


_PAIRS = (("W_self", "dW_self"), ("W_neigh", "dW_neigh"), ("b", "db"))


def apply(opt: Optim, params, grads, state1=None, state2=None):
    """Updates every weight (and bias when present) of the model.

    params/state dicts: W_self, W_neigh, b (lists per layer), W_cls, b_cls.
    Returns (new_params, new_state1, new_state2)."""
    def empty():
        return dict(W_self=[], W_neigh=[], b=[], W_cls=None, b_cls=None)

    new, n1, n2 = empty(), empty(), empty()

    def one(W, g, key, idx):
        if W is None:
            return None, None, None
        s1 = None if state1 is None else (state1[key][idx] if idx is not None else state1[key])
        s2 = None if state2 is None else (state2[key][idx] if idx is not None else state2[key])
        return update(opt, W, g, s1, s2)

    L = len(params["W_self"])
    for l in range(L):
        for wk, gk in _PAIRS:
            W = params[wk][l] if params.get(wk) else None
            r = one(W, grads[gk][l] if W is not None else None, wk, l)
            new[wk].append(r[0])
            n1[wk].append(r[1])
            n2[wk].append(r[2])
    for wk, gk in (("W_cls", "dW_cls"), ("b_cls", "db_cls")):
        W = params.get(wk)
        r = one(W, grads.get(gk) if W is not None else None, wk, None)
        new[wk], n1[wk], n2[wk] = r
    return new, n1, n2
