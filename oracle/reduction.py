"""Redundancy reduction (Section 3.2): Algorithms 1-3 applied in rounds.

One round on neighbour lists L_w (w < n, the aggregators):
  Alg. 1  aggregation graph G_a: a pair {x, y} gets weight = number of lists
          that hold both x and y; its attribute set is those lists; pairs of
          weight 1 are dropped.
  Alg. 2  greedy matching: take pairs by decreasing weight while the weight
          exceeds theta; accept a pair only if neither endpoint was taken.
  Alg. 3  each accepted pair {x, y} gets a new vertex v'; every list in the
          pair's attribute set loses x and y and gains v'.
Rounds repeat on the rewritten lists (which may now hold new vertices); the
matchings of all rounds are kept in order, and new vertex ids are contiguous
after n (Section 4.2: ids of a round follow those of the rounds before it).

Readings where the paper is silent (each listed in the design notes):
  * Alg. 1 counts ordered keys (u, w) and (w, u); both count the same lists,
    so the oracle folds them to unordered pairs x < y.
  * Alg. 2's loop condition is a strict "weight > theta".
  * Equal weights are taken in (smaller id, larger id) ascending order.
  * The k-th accepted pair of a round gets id (n + pairs accepted in earlier
    rounds + k), 0-based.
  * Every list is kept sorted ascending after a round (Alg. 3 does not fix the
    position of v' in the list).
  * Optional budget max_aux: a pair is accepted only while the total number of
    new vertices is below max_aux (the experiments cap sum |M| below B|V_s|,
    Section 6.2); once the budget is exhausted no further round runs.
  * New vertices have empty lists: they are computed from their pair, never
    aggregated.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------- Algorithm 1

def pair_weights(rows, ncols):
    """Algorithm 1 weights for every pair with weight >= 2.

    Returns (x, y, w) int64 arrays, x < y, sorted by (x, y). Counting every
    unordered pair of every list uses np.unique as the hash table.
    """
    keys = []
    for L in rows:
        d = len(L)
        if d < 2:
            continue
        arr = np.asarray(L, dtype=np.int64)   # sorted ascending
        i, j = np.triu_indices(d, 1)
        keys.append(arr[i] * ncols + arr[j])
    if not keys:
        z = np.zeros(0, np.int64)
        return z, z, z
    uk, cnt = np.unique(np.concatenate(keys), return_counts=True)
    keep = cnt >= 2
    uk, cnt = uk[keep], cnt[keep].astype(np.int64)
    return uk // ncols, uk % ncols, cnt


def aggregation_graph_literal(rows):
    """Algorithm 1 as written: hash tables keyed by ordered pairs (u, w).

    Returns (W_a, D_a) dicts keyed by unordered (x, y), x < y, after dropping
    weight-1 pairs. Only for small graphs (pure Python loops).
    """
    W, D = {}, {}
    for v, L in enumerate(rows):
        for u in L:
            for w in L:
                if w == u:
                    continue
                W[(u, w)] = W.get((u, w), 0) + 1
                D.setdefault((u, w), set()).add(v)
    Wf, Df = {}, {}
    for (u, w), c in W.items():
        if c == 1:
            continue
        key = (min(u, w), max(u, w))
        # (u, w) and (w, u) hold the same count and attribute set
        if key in Wf:
            assert Wf[key] == c and Df[key] == D[(u, w)]
        Wf[key] = c
        Df[key] = D[(u, w)]
    return Wf, Df


# ---------------------------------------------------------------- Algorithm 2

def greedy_matching(x, y, w, theta, nverts, budget_left=None):
    """Algorithm 2: scan pairs by decreasing weight while weight > theta.

    Equal weights are ordered by (x, y) ascending. A pair is accepted when both
    endpoints are still free (and, with a budget, while budget remains).
    Returns the accepted pairs in acceptance order as a list of (x, y, weight),
    and whether the budget ran out.
    """
    cand = w > theta
    x, y, w = x[cand], y[cand], w[cand]
    order = np.lexsort((y, x, -w))
    free = np.ones(nverts, dtype=bool)
    out = []
    exhausted = False
    for k in order:
        if budget_left is not None and len(out) >= budget_left:
            exhausted = True
            break
        a, b = int(x[k]), int(y[k])
        if not (free[a] and free[b]):
            continue
        free[a] = free[b] = False
        out.append((a, b, int(w[k])))
    return out, exhausted


# ---------------------------------------------------------------- Algorithm 3

def rewrite(rows, matched, first_id):
    """Algorithm 3: the j-th matched pair {x, y} becomes vertex first_id + j;
    every list holding both x and y swaps them for the new vertex."""
    partner = {}
    for j, (a, b, _) in enumerate(matched):
        partner[a] = (b, first_id + j)
        partner[b] = (a, first_id + j)
    out = []
    for L in rows:
        s = set(L)
        new = []
        for c in L:
            if c in partner:
                p, nid = partner[c]
                if p in s:
                    if c < p:
                        new.append(nid)
                    continue
            new.append(c)
        out.append(sorted(new))
    return out


# ---------------------------------------------------------------- rounds

def num_read(rows):
    """numRead(G) = sum_v d_v (Section 3.2)."""
    return int(sum(len(L) for L in rows))


def num_add(rows):
    """numAdd(G) = sum over d_v >= 1 of (d_v - 1) (Section 3.2)."""
    return int(sum(len(L) - 1 for L in rows if len(L) >= 1))


def reduce(rowptr, col, theta=2, max_rounds=5, max_aux=-1, literal=False):
    """Iterative redundancy reduction of G_s into G_s^# (Section 3.2).

    Returns a dict with
      rowptr, col      CSR of G_s^# over the n aggregators (sorted lists)
      pairs            int64[naux, 2], smaller id first, in id order
      round_offsets    int64[rounds + 1]; pairs of round r are
                       pairs[round_offsets[r]:round_offsets[r+1]]
      stats            per round (|M|, sum of weights, nnz after, numAdd after)
    """
    n = len(rowptr) - 1
    rows = [list(map(int, col[rowptr[w]:rowptr[w + 1]])) for w in range(n)]
    pairs = []
    offsets = [0]
    stats = []
    ncols = n
    for _ in range(max_rounds):
        budget_left = None if max_aux < 0 else max_aux - len(pairs)
        if budget_left is not None and budget_left <= 0:
            break
        if literal:
            Wa, _ = aggregation_graph_literal(rows)
            keys = sorted(Wa)
            x = np.array([k[0] for k in keys], dtype=np.int64)
            y = np.array([k[1] for k in keys], dtype=np.int64)
            w = np.array([Wa[k] for k in keys], dtype=np.int64)
        else:
            x, y, w = pair_weights(rows, ncols)
        matched, exhausted = greedy_matching(x, y, w, theta, ncols, budget_left)
        if not matched:
            break
        rows = rewrite(rows, matched, ncols)
        pairs.extend((a, b) for a, b, _ in matched)
        ncols += len(matched)
        offsets.append(len(pairs))
        stats.append((len(matched), sum(m[2] for m in matched),
                      num_read(rows), num_add(rows)))
        if exhausted:
            break
    out_rowptr = np.zeros(n + 1, dtype=np.int64)
    for i, L in enumerate(rows):
        out_rowptr[i + 1] = out_rowptr[i] + len(L)
    out_col = np.array([c for L in rows for c in L], dtype=np.int64)
    return dict(rowptr=out_rowptr, col=out_col,
                pairs=np.array(pairs, dtype=np.int64).reshape(-1, 2),
                round_offsets=np.array(offsets, dtype=np.int64),
                stats=stats, n=n, naux=len(pairs))


def gammas(rowptr, col, red):
    """gamma_read and gamma_add of Section 3.2 for a reduction result."""
    n = len(rowptr) - 1
    rows0 = [col[rowptr[w]:rowptr[w + 1]] for w in range(n)]
    rows1 = [red["col"][red["rowptr"][w]:red["rowptr"][w + 1]] for w in range(n)]
    m = red["naux"]
    g_read = (num_read(rows1) + 2 * m) / max(num_read(rows0), 1)
    g_add = (num_add(rows1) + m) / max(num_add(rows0), 1)
    return g_read, g_add


def expand(c, n, pairs):
    """Original vertices summed into column c of G_s^# (c itself if c < n)."""
    if c < n:
        return [c]
    a, b = pairs[c - n]
    return expand(int(a), n, pairs) + expand(int(b), n, pairs)
