"""Subgraph construction for the oracle.

The GCN input is an undirected graph; A is its 0/1 adjacency and D the
diagonal degree matrix (Section 2.1, text around Eq. 1). A minibatch is the
subgraph induced on a sampled vertex set, with the same vertex set used by
every layer (Section 3.1, "Minibatch by sampling training graph").
"""
from __future__ import annotations

import numpy as np


class GraphError(ValueError):
    pass


def subgraph_build(n_full, src, dst, vertices=None):
    """Induced, undirected, simple subgraph in CSR form.

    Edges (src[i], dst[i]) are read as undirected. If `vertices` is given the
    subgraph is induced on it and vertex vertices[k] becomes k; otherwise all
    n_full vertices are kept. Self-loops and repeated edges are dropped (A is
    0/1 and D counts neighbours). Neighbour lists are sorted ascending.

    Returns (rowptr int64[n+1], col int64[nnz]).
    """
    src = np.asarray(src, dtype=np.int64).ravel()
    dst = np.asarray(dst, dtype=np.int64).ravel()
    if src.shape != dst.shape:
        raise GraphError("src and dst differ in length")
    if n_full < 0:
        raise GraphError("negative vertex count")
    if src.size and (src.min() < 0 or dst.min() < 0 or src.max() >= n_full
                     or dst.max() >= n_full):
        raise GraphError("edge endpoint out of range")
    if vertices is None:
        n = int(n_full)
        relabel = {v: v for v in range(n)}
    else:
        vertices = [int(v) for v in vertices]
        if any(v < 0 or v >= n_full for v in vertices):
            raise GraphError("vertex id out of range")
        if len(set(vertices)) != len(vertices):
            raise GraphError("repeated vertex in subset")
        n = len(vertices)
        relabel = {v: k for k, v in enumerate(vertices)}
    neigh = [set() for _ in range(n)]
    for u, v in zip(src.tolist(), dst.tolist()):
        if u == v:
            continue
        if u in relabel and v in relabel:
            a, b = relabel[u], relabel[v]
            neigh[a].add(b)
            neigh[b].add(a)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    for w in range(n):
        rowptr[w + 1] = rowptr[w] + len(neigh[w])
    col = np.zeros(int(rowptr[-1]), dtype=np.int64)
    for w in range(n):
        col[rowptr[w]:rowptr[w + 1]] = sorted(neigh[w])
    return rowptr, col


def degrees(rowptr):
    """d_v = |N(v)| (the diagonal of D)."""
    return np.diff(np.asarray(rowptr, dtype=np.int64))


def inv_degrees(rowptr):
    """1/d_v, and 0 for an isolated vertex (whose aggregated row is zero)."""
    d = degrees(rowptr).astype(np.float64)
    out = np.zeros_like(d)
    nz = d > 0
    out[nz] = 1.0 / d[nz]
    return out


def rows_of(rowptr, col):
    """Neighbour lists as Python lists."""
    return [list(map(int, col[rowptr[w]:rowptr[w + 1]]))
            for w in range(len(rowptr) - 1)]


def adjacency_dense(rowptr, col, ncols=None):
    """Dense 0/1 matrix with A[w, c] = 1 for c in row w (float64)."""
    n = len(rowptr) - 1
    A = np.zeros((n, n if ncols is None else ncols), dtype=np.float64)
    for w in range(n):
        for c in col[rowptr[w]:rowptr[w + 1]]:
            A[w, c] += 1.0
    return A
