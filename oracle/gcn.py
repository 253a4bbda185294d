"""GCN training step for the oracle, float64 throughout.

Layer l (Eq. 1):   H_l = ReLU( H_{l-1} W_self | D^-1 A H_{l-1} W_neigh )
                   ("|" concatenates column-wise, self branch first).
Classifier:        logits = H_L W_cls (+ b_cls), linear (a ReLU in front of a
                   softmax would clip the logits; Section 2.1 writes the MLP
                   layer with a ReLU, read here as the hidden-layer form).
Loss:              softmax cross-entropy, mean over the n vertices, or
                   sigmoid binary cross-entropy, mean over the n*C entries.
Backward (Eq. 2a-2c), G = mask(dL/dH_l) with mask = ReLU' (0 at 0):
                   dW_self  = H_{l-1}^T G[:, :h]
                   dW_neigh = (D^-1 A H_{l-1})^T G[:, h:]
                   dH_{l-1} = G[:, :h] W_self^T + A D^-1 G[:, h:] W_neigh^T
Update:            W <- W - lr dW (plain gradient descent, Section 4.1 notes
                   vanilla gradient descent keeps no optimiser state); momentum
                   and Adam in optim.py.

Optional biases (not in Eq. 1; kept off by default): b_l in R^{2h} added
before the ReLU, b_cls in R^C added to the logits.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

from . import graph as _graph
from . import optim as _optim

SOFTMAX_CE = 0
SIGMOID_BCE = 1


def adjacency(rowptr, col, n):
    """A as a SciPy CSR matrix (0/1, float64)."""
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    data = np.ones(col.size, dtype=np.float64)
    return sp.csr_matrix((data, col, rowptr), shape=(n, n))


# ---------------------------------------------------------------- aggregation

def aggregate(rowptr, col, H):
    """Feature aggregation D^-1 A H: row w is the mean of its neighbours'
    rows (Section 2.1, Eq. 1); an isolated vertex gets a zero row."""
    H = np.asarray(H, dtype=np.float64)
    n = len(rowptr) - 1
    A = adjacency(rowptr, col, n)
    return _graph.inv_degrees(rowptr)[:, None] * (A @ H)


def aggregate_transposed(rowptr, col, G):
    """A D^-1 G, the aggregation in the input-gradient term of Eq. 2c."""
    G = np.asarray(G, dtype=np.float64)
    n = len(rowptr) - 1
    A = adjacency(rowptr, col, n)
    return A @ (_graph.inv_degrees(rowptr)[:, None] * G)


def aux_rows(red, H):
    """Pre-computed pair sums X_M (Section 4.2 step 1), round by round:
    row k is the sum of the rows of its pair's two vertices, where a vertex
    id >= n refers to an earlier pair sum."""
    H = np.asarray(H, dtype=np.float64)
    n = H.shape[0]
    ext = np.zeros((n + red["naux"], H.shape[1]), dtype=np.float64)
    ext[:n] = H
    for k, (a, b) in enumerate(red["pairs"]):
        ext[n + k] = ext[a] + ext[b]
    return ext[n:]


def aggregate_reduced(red, inv_deg, H, scale="post"):
    """Aggregation on G_s^# in the three steps of Section 4.2: pair sums,
    then A^# times the extended features, then the degree scaling.

    scale="post": D^-1 (A^# X_ext)  (forward aggregation)
    scale="pre" : A^# (D^-1 X)_ext  (the A D^-1 term of Eq. 2c)
    """
    H = np.asarray(H, dtype=np.float64)
    inv_deg = np.asarray(inv_deg, dtype=np.float64)
    n = H.shape[0]
    src = inv_deg[:, None] * H if scale == "pre" else H
    ext = np.concatenate([src, aux_rows(red, src)], axis=0)
    out = np.zeros_like(H)
    rp, cl = red["rowptr"], red["col"]
    for w in range(n):
        for c in cl[rp[w]:rp[w + 1]]:
            out[w] += ext[c]
    if scale == "post":
        out *= inv_deg[:, None]
    return out


# ---------------------------------------------------------------- loss

def softmax_ce(logits, labels):
    """Mean softmax cross-entropy and dL/dlogits = (softmax - onehot) / n."""
    z = np.asarray(logits, dtype=np.float64)
    n = z.shape[0]
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(s[:, 0])
    y = np.asarray(labels, dtype=np.int64)
    loss = float(np.mean(lse - z[np.arange(n), y]))
    dz = e / s
    dz[np.arange(n), y] -= 1.0
    return loss, dz / n


def sigmoid_bce(logits, labels):
    """Mean binary cross-entropy of sigmoid(logits) against 0/1 labels over
    all n*C entries, and dL/dlogits = (sigmoid - y) / (n C)."""
    z = np.asarray(logits, dtype=np.float64)
    y = np.asarray(labels, dtype=np.float64)
    per = np.maximum(z, 0.0) - z * y + np.log1p(np.exp(-np.abs(z)))
    sig = 0.5 * (1.0 + np.tanh(0.5 * z))   # logistic function, overflow-free
    return float(per.mean()), (sig - y) / z.size


def loss_and_grad(kind, logits, labels):
    if kind == SOFTMAX_CE:
        return softmax_ce(logits, labels)
    if kind == SIGMOID_BCE:
        return sigmoid_bce(logits, labels)
    raise ValueError("unknown loss")


# ---------------------------------------------------------------- model

def forward(rowptr, col, X, params):
    """Eq. 1 for every layer, then the classifier.

    params: dict with lists W_self, W_neigh, b (entries may be None) and
    W_cls, b_cls (may be None). Returns a dict of all activations.
    """
    H = np.asarray(X, dtype=np.float64)
    Hs, AHs, Zs = [H], [], []
    L = len(params["W_self"])
    for l in range(L):
        Ws = np.asarray(params["W_self"][l], dtype=np.float64)
        Wn = np.asarray(params["W_neigh"][l], dtype=np.float64)
        AH = aggregate(rowptr, col, H)
        Z = np.concatenate([H @ Ws, AH @ Wn], axis=1)
        b = params["b"][l] if params.get("b") else None
        if b is not None:
            Z = Z + np.asarray(b, dtype=np.float64)[None, :]
        H = np.maximum(Z, 0.0)
        AHs.append(AH)
        Zs.append(Z)
        Hs.append(H)
    logits = H @ np.asarray(params["W_cls"], dtype=np.float64)
    if params.get("b_cls") is not None:
        logits = logits + np.asarray(params["b_cls"], dtype=np.float64)[None, :]
    return dict(H=Hs, AH=AHs, Z=Zs, logits=logits)


def backward(rowptr, col, params, fw, dlogits, masks=None):
    """Eq. 2a-2c for every layer, plus the classifier's gradients.

    masks: optional list of 0/1 arrays, one per layer, to use as the ReLU
    decision instead of [Z_l > 0]. By default the decision is this oracle's
    own, from its float64 Z_l. A caller comparing with a lower-precision
    computation may override entries whose |Z_l| lies within that
    computation's rounding of zero (the caller states and checks the bound).

    Returns dict with dW_self, dW_neigh, db (lists, layer order), dW_cls,
    db_cls, G (masked gradients per layer) and dH (dL/dH_l for l = 1..L).
    """
    L = len(params["W_self"])
    dZc = np.asarray(dlogits, dtype=np.float64)
    Wc = np.asarray(params["W_cls"], dtype=np.float64)
    out = dict(dW_self=[None] * L, dW_neigh=[None] * L, db=[None] * L,
               G=[None] * L, dH=[None] * L)
    out["dW_cls"] = fw["H"][L].T @ dZc
    out["db_cls"] = dZc.sum(axis=0)
    dH = dZc @ Wc.T
    for l in range(L - 1, -1, -1):
        out["dH"][l] = dH
        mask = fw["Z"][l] > 0.0 if masks is None else np.asarray(masks[l], bool)
        G = dH * mask
        h = G.shape[1] // 2
        Gs, Gn = G[:, :h], G[:, h:]
        out["G"][l] = G
        out["dW_self"][l] = fw["H"][l].T @ Gs
        out["dW_neigh"][l] = fw["AH"][l].T @ Gn
        out["db"][l] = G.sum(axis=0)
        if l > 0:
            Ws = np.asarray(params["W_self"][l], dtype=np.float64)
            Wn = np.asarray(params["W_neigh"][l], dtype=np.float64)
            dH = Gs @ Ws.T + aggregate_transposed(rowptr, col, Gn) @ Wn.T
    return out


def sgd(params, grads, lr):
    """W <- W - lr dW for every weight (and bias when present)."""
    L = len(params["W_self"])
    new = dict(W_self=[], W_neigh=[], b=[], W_cls=None, b_cls=None)
    for l in range(L):
        new["W_self"].append(np.asarray(params["W_self"][l], np.float64)
                             - lr * grads["dW_self"][l])
        new["W_neigh"].append(np.asarray(params["W_neigh"][l], np.float64)
                              - lr * grads["dW_neigh"][l])
        b = params["b"][l] if params.get("b") else None
        new["b"].append(None if b is None else
                        np.asarray(b, np.float64) - lr * grads["db"][l])
    new["W_cls"] = np.asarray(params["W_cls"], np.float64) - lr * grads["dW_cls"]
    if params.get("b_cls") is not None:
        new["b_cls"] = np.asarray(params["b_cls"], np.float64) - lr * grads["db_cls"]
    return new


def train_step(rowptr, col, X, params, labels, loss_kind, lr, masks=None, opt=None,
               state1=None, state2=None, fw=None):
    """One forward + loss + backward + update step: plain gradient descent
    with step lr, or the optimiser `opt` (optim.Optim) with its states.
    fw: forward() of these same inputs, when already computed."""
    if fw is None:
        fw = forward(rowptr, col, X, params)
    loss, dlogits = loss_and_grad(loss_kind, fw["logits"], labels)
    grads = backward(rowptr, col, params, fw, dlogits, masks)
    if opt is None:
        return dict(fw=fw, loss=loss, dlogits=dlogits, grads=grads,
                    params=sgd(params, grads, lr))
    new, s1, s2 = _optim.apply(opt, params, grads, state1, state2)
    return dict(fw=fw, loss=loss, dlogits=dlogits, grads=grads, params=new, state1=s1,
                state2=s2)


def loss_only(rowptr, col, X, params, labels, loss_kind):
    fw = forward(rowptr, col, X, params)
    return loss_and_grad(loss_kind, fw["logits"], labels)[0]
