"""Top-K expert routing and the token -> expert permutation.

Rollout routing replay records the expert choices made during generation so the
actor can reuse them (Sec. 4.1; the expert-route records travel with each
experience, Sec. 4.4). The route record is the top-K expert IDs per token per
MoE layer. The router's rules, in the method's reading:
  * router logits g = y W_r^T (+ optional bias) in float32;
  * top-K by descending logit, ties to the lower expert ID, -0.0 equal to +0.0;
  * weights = softmax over the K selected logits (equal to the full softmax
    renormalised over the selection).
The permutation groups the T*K (token, slot) pairs by expert, stably: order by
(expert, token, slot). counts[e], offsets = exclusive prefix sum, perm[r] = the
pair index t*K + j placed at row r, inv[t*K + j] = its row.
"""
import numpy as np


def router_logits_f32(y, w_router, bias=None):
    """float64 dot products rounded once to float32 (the correctly rounded value)."""
    g = np.asarray(y, dtype=np.float64) @ np.asarray(w_router, dtype=np.float64).T
    g = g.astype(np.float32)
    if bias is not None:
        g = (g + np.asarray(bias, dtype=np.float32)).astype(np.float32)
    return g


def topk_route(logits, K):
    """logits [T, E] float32 -> ids [T, K] int32, weights [T, K] float32, margin [T],
    order_margin [T].

    margin[t] = gap between the K-th and (K+1)-th logits (inf if K == E): below it, the
    selected set can change under last-bit differences in the logits. order_margin[t] =
    smallest gap between adjacent selected logits: below it, the slot order can."""
    g = np.asarray(logits, dtype=np.float32)
    T, E = g.shape
    ids = np.zeros((T, K), dtype=np.int32)
    wts = np.zeros((T, K), dtype=np.float32)
    margin = np.full(T, np.inf)
    order_margin = np.full(T, np.inf)
    for t in range(T):
        row = g[t].astype(np.float64) + 0.0       # -0.0 -> +0.0
        order = sorted(range(E), key=lambda e: (-row[e], e))
        sel = order[:K]
        ids[t] = sel
        vals = row[sel]
        ev = np.exp(vals - vals.max())
        wts[t] = (ev / ev.sum()).astype(np.float32)
        if K < E:
            margin[t] = row[order[K - 1]] - row[order[K]]
        if K > 1:
            order_margin[t] = float(np.min(vals[:-1] - vals[1:]))
    return ids, wts, margin, order_margin


def permute(ids, E):
    """Stable grouping of (token, slot) pairs by expert."""
    ids = np.asarray(ids)
    T, K = ids.shape
    flat = ids.reshape(-1)
    counts = np.bincount(flat, minlength=E).astype(np.int32)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    perm = np.zeros(T * K, dtype=np.int32)
    inv = np.zeros(T * K, dtype=np.int32)
    fill = offsets[:-1].copy()
    for p in range(T * K):          # pairs visited in (token, slot) order
        e = flat[p]
        perm[fill[e]] = p
        inv[p] = fill[e]
        fill[e] += 1
    return counts, offsets, perm, inv
