"""Independent reference computations used to pin the oracle.

None of these retypes the oracle's formulas: each goes through a different
route that the paper's mathematics fixes to the same answer.

* nearest-codeword assignment through ``scipy.spatial.distance.cdist`` and a
  stable argsort (lowest index on exact ties);
* aggregates through ``numpy.add.at`` / ``bincount``;
* attention through ``torch.nn.functional.scaled_dot_product_attention`` in
  fp64 over the per-key quantised keys (the regrouping identity of Sec. 3.2
  and the replacement identity of App. C say the codeword-level sums equal
  per-key attention over quantised keys);
* top-P through exhaustive enumeration of all P-subsets.
"""
from __future__ import annotations

import itertools

import numpy as np
import torch
from scipy.spatial.distance import cdist


def nearest(points: np.ndarray, codes: np.ndarray):
    """Index of the nearest code (squared L2, lowest index on ties) and the
    sorted distances, via scipy cdist."""
    D = cdist(points, codes, metric="sqeuclidean")
    order = np.argsort(D, axis=1, kind="stable")
    return order[:, 0], np.take_along_axis(D, order, axis=1)


def tree_assign(K, Cp, Cc):
    """Per key: nearest parent, then nearest child of that parent, moving only
    when the child is strictly closer (Alg. 1)."""
    B, H, N, d = K.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    par = np.empty((B, H, N), np.int64)
    code = np.empty((B, H, N), np.int64)
    for b in range(B):
        for h in range(H):
            p, Dp = nearest(K[b, h], Cp[h])
            par[b, h] = p
            for j in range(N):
                c, Dc = nearest(K[b, h, j][None], Cc[h, p[j]])
                moved = Dc[0, 0] < Dp[j, 0]
                code[b, h, j] = M0 + p[j] * Ch + c[0] if moved else p[j]
    return par, code


def aggregates(V, par, code, M0, Ch):
    B, H, N, d = V.shape
    Mtot = M0 * (1 + Ch)
    Vbar = np.zeros((B, H, Mtot, d))
    n = np.zeros((B, H, Mtot), np.int64)
    for b in range(B):
        for h in range(H):
            np.add.at(Vbar[b, h], par[b, h], V[b, h])
            n[b, h] += np.bincount(par[b, h], minlength=Mtot)
            moved = code[b, h] >= M0
            np.add.at(Vbar[b, h], code[b, h][moved], V[b, h][moved])
            n[b, h] += np.bincount(code[b, h][moved], minlength=Mtot)
    return Vbar, n


def sdpa(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Softmax attention with logits exactly q.k (scale 1), fp64 on the CPU."""
    tq = torch.from_numpy(np.ascontiguousarray(q))[None, None]
    tk = torch.from_numpy(np.ascontiguousarray(k))[None, None]
    tv = torch.from_numpy(np.ascontiguousarray(v))[None, None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=1.0)
    return out[0, 0].numpy()


def attention_probs(q: np.ndarray, k: np.ndarray) -> np.ndarray:
    tq = torch.from_numpy(np.ascontiguousarray(q))
    tk = torch.from_numpy(np.ascontiguousarray(k))
    return torch.softmax(tq @ tk.T, dim=-1).numpy()


def quantised_keys(Cp, Cc, par, code, selected=None):
    """Per-key codeword under App. C's replacement: a key that moved to a child
    of a selected parent is represented by that child, every other key by its
    parent. ``selected=None`` means every parent is selected."""
    M0, Ch = Cc.shape[0], Cc.shape[1]
    khat = Cp[par].copy()
    moved = code >= M0
    if selected is not None:
        moved &= np.isin(par, np.asarray(selected))
    cidx = code[moved] - M0
    khat[moved] = Cc[cidx // Ch, cidx % Ch]
    return khat


def per_key_importance(Q, Cp, par):
    """w_a(I) as the softmax mass that the queries of I put on the keys of
    parent cell a, with every key replaced by its parent (per-key route)."""
    probs = attention_probs(Q, Cp[par])
    M0 = Cp.shape[0]
    return np.stack([np.bincount(par, weights=probs[i], minlength=M0)
                     for i in range(Q.shape[0])]).sum(axis=0)


def topp_by_enumeration(w: np.ndarray, P: int):
    """Exhaustive search over all P-subsets: the subset whose importances,
    sorted in decreasing order, are lexicographically largest (so every rank
    holds the largest value any subset can put there, hence also the largest
    total); among subsets with equal sorted importances, the one whose sorted
    index tuple is smallest. Returned in the canonical order (w desc, index
    asc)."""
    M0 = len(w)
    best, best_key = None, None
    for sub in itertools.combinations(range(M0), P):
        vals = sorted((-w[a], a) for a in sub)
        key = (tuple(v for v, _ in vals), tuple(sub))
        if best_key is None or key < best_key:
            best_key, best = key, [a for _, a in vals]
    return np.array(best, np.int64)


def hilbert_cells(n: int):
    """Cells (x, y) of the Hilbert curve of an n x n grid (n a power of two),
    in curve order: the textbook conversion of a curve index to a cell, which
    reads the index two bits at a time from the lowest, rotating or reflecting
    the partial cell in each quadrant."""
    xs = np.empty(n * n, np.int64)
    ys = np.empty(n * n, np.int64)
    for t0 in range(n * n):
        t, x, y, s = t0, 0, 0, 1
        while s < n:
            rx = 1 & (t // 2)
            ry = 1 & (t ^ rx)
            if ry == 0:
                if rx == 1:
                    x, y = s - 1 - x, s - 1 - y
                x, y = y, x
            x += s * rx
            y += s * ry
            t //= 4
            s *= 2
        xs[t0], ys[t0] = x, y
    return xs, ys

