"""Seeded synthetic workloads shaped like the paper's subgraph minibatches.

This module only draws inputs: graphs, features, weights and labels. It holds
none of the method's arithmetic (no aggregation, no reduction, no GCN maths),
so both the HIP path and the CPU oracle can take their inputs from it.

The paper trains on subgraphs induced from PPI, Reddit and Yelp (Section 6,
Table 2: attribute lengths 50 / 602 / 300, 121 / 41 / 100 classes). Those
datasets are not available here; the workloads below are Chung-Lu random
graphs with power-law expected degrees standing in for the sampled subgraphs,
with the datasets' feature widths, class counts and label kinds.

Recipe (every workload):
  * seed = SeedSequence([workload_id]) (or [5, i] for the i-th subgraph of the
    epoch-shaped stream); four PCG64 child streams: graph, features, weights,
    labels, in that order.
  * Chung-Lu: raw weights r_i = (i+1)^(-1/(gamma-1)), S = sum(r),
    p_ij = min(1, c r_i r_j / S) for i < j, with c found by bisection so the
    expected edge count is n*dbar/2; one Bernoulli draw per pair, row by row;
    then a seeded random relabelling so that hubs are not the low ids.
    No self-loops; each undirected edge listed once.
  * features ~ N(0, 1) float32, n x f_in.
  * Glorot-uniform float32 weights, bound sqrt(6 / (fan_in + fan_out)), drawn in
    the order W_self(1), W_neigh(1), ..., W_self(L), W_neigh(L), W_cls.
  * labels: uniform class ids (int32) for softmax cross-entropy; Bernoulli(p)
    multi-hot uint8 rows for sigmoid binary cross-entropy.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

SOFTMAX_CE = 0
SIGMOID_BCE = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one subgraph training step."""
    name: str
    n: int            # subgraph vertices |V_s|
    gamma: float      # power-law exponent of the expected degrees
    dbar: float       # target mean degree
    L: int            # graph convolutional layers
    f_in: int         # input attribute length f^(0)
    h: int            # width of each branch (layer output is 2h wide)
    C: int            # classes
    loss: int         # SOFTMAX_CE or SIGMOID_BCE
    label_p: float = 0.0      # Bernoulli rate of multi-hot labels
    reduce: bool = True       # aggregation on the redundancy-reduced graph
    theta: int = 2            # greedy-matching threshold
    rounds: int = 5           # reduction rounds
    budget: float = -1.0      # aux budget B: sum |M| < B * n (negative: none)
    lr: float = 0.01
    seed: tuple = ()

    @property
    def max_aux(self) -> int:
        if self.budget < 0:
            return -1
        return int(math.ceil(self.budget * self.n)) - 1


# The five workloads: a tiny smoke case, three stand-ins with the PPI / Reddit /
# Yelp attribute and class widths, and one subgraph of the epoch-shaped stream.
WORKLOADS = {
    "tiny": Workload("tiny", 1024, 2.5, 10, 2, 64, 128, 16, SOFTMAX_CE,
                     reduce=True, seed=(1,)),
    "ppi8k": Workload("ppi8k", 8000, 2.5, 15, 2, 50, 512, 121, SIGMOID_BCE,
                      label_p=0.1, reduce=True, budget=2.0, seed=(2,)),
    "reddit8k": Workload("reddit8k", 8000, 2.2, 30, 2, 602, 128, 41, SOFTMAX_CE,
                         reduce=False, budget=0.5, seed=(3,)),
    "yelp10k": Workload("yelp10k", 10000, 2.5, 20, 3, 300, 512, 100, SIGMOID_BCE,
                        label_p=0.05, reduce=True, budget=0.5, seed=(4,)),
    "stream8k": Workload("stream8k", 8000, 2.5, 20, 3, 256, 256, 64, SOFTMAX_CE,
                         reduce=True, budget=0.5, seed=(5, 0)),
}
STREAM_LEN = 64


def stream_workload(i: int) -> Workload:
    """The i-th independently seeded subgraph of the 64-step stream."""
    return dataclasses.replace(WORKLOADS["stream8k"], seed=(5, int(i)))


def _streams(seed):
    ss = np.random.SeedSequence(list(seed))
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]


def _expected_edges(c, r, S):
    """sum_{i<j} min(1, c r_i r_j / S) for r sorted in decreasing order."""
    a = c * r / S                       # row i contributes sum_j min(1, a_i r_j)
    neg = -r                            # ascending copy for searchsorted
    csum = np.concatenate([[0.0], np.cumsum(r)])
    # number of j with a_i r_j >= 1  <=>  r_j >= 1/a_i
    t = np.searchsorted(neg, -1.0 / a, side="right")
    full = t + a * (csum[-1] - csum[t])
    diag = np.minimum(1.0, a * r)
    return 0.5 * (full.sum() - diag.sum())


def chung_lu_edges(n, gamma, dbar, rng):
    """Undirected Chung-Lu edge list (src < dst before relabelling)."""
    r = (np.arange(n, dtype=np.float64) + 1.0) ** (-1.0 / (gamma - 1.0))
    S = r.sum()
    target = n * dbar / 2.0
    lo, hi = 0.0, 1.0
    while _expected_edges(hi, r, S) < target:
        hi *= 2.0
        if hi > 1e12:
            raise ValueError("mean degree not reachable")
    for _ in range(100):
        mid = 0.5 * (lo + hi)
        if _expected_edges(mid, r, S) < target:
            lo = mid
        else:
            hi = mid
    c = 0.5 * (lo + hi)
    src, dst = [], []
    for i in range(n - 1):
        p = np.minimum(1.0, (c * r[i] / S) * r[i + 1:])
        hit = np.nonzero(rng.random(n - 1 - i) < p)[0]
        if hit.size:
            src.append(np.full(hit.size, i, np.int64))
            dst.append(hit.astype(np.int64) + i + 1)
    src = np.concatenate(src) if src else np.zeros(0, np.int64)
    dst = np.concatenate(dst) if dst else np.zeros(0, np.int64)
    perm = rng.permutation(n).astype(np.int64)
    return perm[src], perm[dst]


def glorot(rng, fan_in, fan_out):
    a = math.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-a, a, size=(fan_in, fan_out)).astype(np.float32)


@dataclasses.dataclass
class Inputs:
    wl: Workload
    src: np.ndarray          # int64 [m] undirected edges
    dst: np.ndarray          # int64 [m]
    X: np.ndarray            # float32 [n, f_in]
    W_self: list             # float32 [F_l, h] per layer
    W_neigh: list            # float32 [F_l, h] per layer
    W_cls: np.ndarray        # float32 [2h, C]
    labels: np.ndarray       # int32 [n] or uint8 [n, C]


def layer_in_width(wl: Workload, layer: int) -> int:
    """Input width of 1-based layer `layer`."""
    return wl.f_in if layer == 1 else 2 * wl.h


def make_inputs(wl: Workload) -> Inputs:
    g_rng, x_rng, w_rng, y_rng = _streams(wl.seed)
    src, dst = chung_lu_edges(wl.n, wl.gamma, wl.dbar, g_rng)
    X = x_rng.standard_normal((wl.n, wl.f_in), dtype=np.float32)
    Ws, Wn = [], []
    for layer in range(1, wl.L + 1):
        F = layer_in_width(wl, layer)
        Ws.append(glorot(w_rng, F, wl.h))
        Wn.append(glorot(w_rng, F, wl.h))
    Wc = glorot(w_rng, 2 * wl.h, wl.C)
    if wl.loss == SOFTMAX_CE:
        labels = y_rng.integers(0, wl.C, size=wl.n).astype(np.int32)
    else:
        labels = (y_rng.random((wl.n, wl.C)) < wl.label_p).astype(np.uint8)
    return Inputs(wl, src, dst, X, Ws, Wn, Wc, labels)


def small_workload(n, dbar, L, f_in, h, C, loss, seed, gamma=2.5, reduce=True,
                   theta=2, rounds=5, label_p=0.2, budget=-1.0) -> Workload:
    """Ad-hoc workload for parity cases at sizes the oracle finishes quickly."""
    return Workload(f"n{n}_f{f_in}_h{h}_c{C}", n, gamma, dbar, L, f_in, h, C,
                    loss, label_p=label_p, reduce=reduce, theta=theta,
                    rounds=rounds, budget=budget, seed=(1000,) + tuple(seed))


def chung_lu_edge_draws(n, gamma, dbar, rng):
    """Chung-Lu graph for full training graphs too large for one draw per
    pair: round(n dbar / 2) edges, each endpoint drawn independently with
    probability r_i / sum(r) (the same raw weights as chung_lu_edges), then a
    seeded relabelling. Self-loops and repeated edges stay in the list; the
    graph builders drop them, so the realised mean degree is a little below
    dbar."""
    r = (np.arange(n, dtype=np.float64) + 1.0) ** (-1.0 / (gamma - 1.0))
    cdf = np.cumsum(r)
    cdf /= cdf[-1]
    m = int(round(n * dbar / 2.0))
    src = np.minimum(np.searchsorted(cdf, rng.random(m), side="right"), n - 1)
    dst = np.minimum(np.searchsorted(cdf, rng.random(m), side="right"), n - 1)
    perm = rng.permutation(n).astype(np.int64)
    return perm[src.astype(np.int64)], perm[dst.astype(np.int64)]


@dataclasses.dataclass(frozen=True)
class SampledWorkload:
    """Minibatches sampled from one full training graph (Section 3.1): the
    full graph's shape, the frontier sampler's size and budget, and the model
    trained on each induced subgraph."""
    name: str
    n_full: int
    gamma: float
    dbar: float
    m: int             # frontier size
    budget: int        # sampled vertices per minibatch
    max_steps: int     # walk cap
    L: int
    f_in: int
    h: int
    C: int
    loss: int
    theta: int = 2
    rounds: int = 5
    aux_budget: float = 0.5
    lr: float = 0.01
    seed: tuple = ()

    @property
    def max_aux(self) -> int:
        return int(math.ceil(self.aux_budget * self.budget)) - 1

    def sample_seed(self, i: int) -> int:
        """Seed of the i-th minibatch's walk (64-bit)."""
        ss = np.random.SeedSequence(list(self.seed) + [int(i)])
        return int(ss.generate_state(1, dtype=np.uint64)[0])


# A Yelp-sized full graph (Table 2: 716,847 vertices, 6,977,410 edges) with
# the epoch stream's model (3 layers, 256 inputs, 256 per branch, 64
# classes); 8,000-vertex minibatches by frontier sampling with 1,000 walkers.
SAMPLED = {
    "yelpfull": SampledWorkload("yelpfull", 716847, 2.5, 2 * 6977410 / 716847, 1000, 8000,
                                200000, 3, 256, 256, 64, SOFTMAX_CE, seed=(6,)),
}


@dataclasses.dataclass
class FullInputs:
    wl: SampledWorkload
    src: np.ndarray
    dst: np.ndarray
    X: np.ndarray           # n_full x f_in float32
    W_self: list
    W_neigh: list
    W_cls: np.ndarray
    labels: np.ndarray      # int32[n_full] (softmax) or uint8[n_full, C]


def make_full_inputs(wl: SampledWorkload, n_full=None) -> FullInputs:
    """The full graph, its features and labels, and the model's initial
    weights (streams: graph, features, weights, labels). `n_full` overrides
    the vertex count (same recipe, for tests)."""
    n = wl.n_full if n_full is None else int(n_full)
    g_rng, x_rng, w_rng, y_rng = _streams(wl.seed)
    src, dst = chung_lu_edge_draws(n, wl.gamma, wl.dbar, g_rng)
    X = x_rng.standard_normal((n, wl.f_in), dtype=np.float32)
    Ws, Wn = [], []
    for layer in range(1, wl.L + 1):
        fi = wl.f_in if layer == 1 else 2 * wl.h
        Ws.append(glorot(w_rng, fi, wl.h))
        Wn.append(glorot(w_rng, fi, wl.h))
    Wc = glorot(w_rng, 2 * wl.h, wl.C)
    if wl.loss == SOFTMAX_CE:
        labels = y_rng.integers(0, wl.C, size=n).astype(np.int32)
    else:
        labels = (y_rng.random((n, wl.C)) < 0.1).astype(np.uint8)
    return FullInputs(wl, src, dst, X, Ws, Wn, Wc, labels)


def random_edges(n, m, rng, self_loops=True, duplicates=True):
    """Uniform random edge list (may hold self-loops and repeats) for tests of
    the subgraph builder's clean-up."""
    src = rng.integers(0, n, size=m).astype(np.int64)
    dst = rng.integers(0, n, size=m).astype(np.int64)
    if not self_loops:
        keep = src != dst
        src, dst = src[keep], dst[keep]
    if duplicates and src.size:
        k = max(1, src.size // 10)
        s0, d0 = src, dst
        src = np.concatenate([s0, d0[:k]])
        dst = np.concatenate([d0, s0[:k]])
    return src, dst
