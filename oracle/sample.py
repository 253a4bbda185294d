"""Minibatch sampling for the oracle: frontier sampling and the induced
subgraph (test infrastructure; see the package docstring).

Section 3.1 ("Minibatch by sampling training graph") forms a minibatch by
drawing a vertex subset V_s from the training graph with a graph sampler and
taking the subgraph induced on it, used by every layer. The paper does not
define a sampler; it names the multi-dimensional random walk of the work it
cites (Ribeiro and Towsley, IMC 2010, "frontier sampling") as one such
sampler. That method, restated:

  * a frontier of m vertices is drawn uniformly at random;
  * each step picks a frontier vertex u with probability deg(u) divided by
    the sum of the frontier's degrees, moves along an edge of u chosen
    uniformly at random to v, and puts v in u's place;
  * the vertices visited form the sample.

Readings where the cited method leaves a choice open (each is one of the
readings listed with the design):
  * the initial frontier holds m distinct vertices (draws that repeat a
    vertex already in it are discarded and drawn again);
  * the sample is the initial frontier plus every vertex a step moves to,
    and sampling stops once it holds `budget` vertices, after `max_steps`
    steps, or when every frontier vertex is isolated (no step can move);
  * random numbers come from one counter-based generator, SplitMix64
    (Steele, Lea and Flood, OOPSLA 2014): output i of seed s mixes
    s + (i + 1) * 0x9E3779B97F4A7C15; a uniform integer in [0, b) is the
    high 64 bits of output * b. Draws are taken in this order: the initial
    frontier's vertex ids, then per step the degree-weighted pick and the
    neighbour index;
  * the degree-weighted pick of a draw r in [0, S) is the first frontier
    slot whose running degree sum exceeds r;
  * the sampled vertex ids are returned in ascending order, so the induced
    subgraph's vertex k is the k-th smallest sampled id.

Plain Python loops: meant for small graphs and short walks.
"""
from __future__ import annotations

import numpy as np

_MASK = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(seed: int, i: int) -> int:
    """Output i (0, 1, ...) of the SplitMix64 sequence of `seed`."""
    z = (seed + (i + 1) * _GAMMA) & _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


class Draws:
    """Consecutive SplitMix64 outputs of one seed, as bounded integers."""

    def __init__(self, seed: int):
        self.seed = int(seed) & _MASK
        self.count = 0

    def below(self, bound: int) -> int:
        """Uniform integer in [0, bound), bound >= 1."""
        x = splitmix64(self.seed, self.count)
        self.count += 1
        return (x * bound) >> 64


def frontier_sample(rowptr, col, m, budget, seed, max_steps, trace=None):
    """Frontier sampling of a vertex set (see the module docstring).

    rowptr, col: CSR of the undirected full graph (rows = neighbour lists).
    m: frontier size, 1 <= m <= budget <= n.
    budget: vertices to sample; max_steps >= 0: walk steps at most.
    trace: if a list, receives (slot, u, v) for every step taken.
    Returns the sampled vertex ids, ascending (a Python list).
    """
    rowptr = [int(x) for x in rowptr]
    col = [int(x) for x in col]
    n = len(rowptr) - 1
    if not (1 <= m <= budget <= n) or max_steps < 0:
        raise ValueError("need 1 <= m <= budget <= n and max_steps >= 0")
    deg = [rowptr[v + 1] - rowptr[v] for v in range(n)]
    draws = Draws(seed)

    frontier = []
    sampled = set()
    while len(frontier) < m:
        v = draws.below(n)
        if v not in sampled:
            frontier.append(v)
            sampled.add(v)

    steps = 0
    while len(sampled) < budget and steps < max_steps:
        total = sum(deg[u] for u in frontier)
        if total == 0:
            break
        r = draws.below(total)
        running = 0
        for slot, u in enumerate(frontier):
            running += deg[u]
            if r < running:
                break
        v = col[rowptr[u] + draws.below(deg[u])]
        frontier[slot] = v
        sampled.add(v)
        steps += 1
        if trace is not None:
            trace.append((slot, u, v))
    return sorted(sampled)


def induce(rowptr, col, vertices):
    """Subgraph induced on `vertices` (Section 3.1): vertex vertices[k]
    becomes k, an edge is kept when both ends are in the set, and each
    neighbour list is sorted ascending. Returns (rowptr, col) as int64."""
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    vertices = [int(v) for v in vertices]
    pos = {v: k for k, v in enumerate(vertices)}
    if len(pos) != len(vertices):
        raise ValueError("repeated vertex")
    out_ptr = [0]
    out_col = []
    for v in vertices:
        row = sorted(pos[int(w)] for w in col[rowptr[v]:rowptr[v + 1]] if int(w) in pos)
        out_col.extend(row)
        out_ptr.append(len(out_col))
    return np.asarray(out_ptr, dtype=np.int64), np.asarray(out_col, dtype=np.int64)
