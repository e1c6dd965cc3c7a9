"""Plain float64 CPU oracle of the budget front-ends GRKV is paired with:
per-unit (ragged) retained budgets, a layer-wise pyramid schedule and a
head-wise adaptive allocation.

TEST INFRASTRUCTURE ONLY, like the other oracle modules: imported by the test
suite, the smoke check and the benchmark's CPU-baseline leg, never by the
product path, and sharing no code with the HIP path.

The paper pairs GRKV with several eviction back-ends (Sec. 2, related work;
Sec. 4, compatibility): PyramidKV gives lower layers more of the cache and
higher layers less, Ada-KV gives more to the heads that need long-range
context, and token-based H2O ranks single tokens by accumulated attention.
The merge is the same for all of them; what changes is each unit's budget c_u
(and, for H2O, the absence of pooling).  Readings, since the paper describes
these methods in one sentence each:

* ragged budgets: every unit is compressed exactly as in ``grkv_oracle`` with
  its own budget c_u (w <= c_u <= n), the fixed set using floor(beta * c_u);
* pyramid: budgets fall linearly from the bottom layer to the top, the top
  layer keeping ``ratio`` (default 1/2) of the mean and the bottom layer
  2 - ratio of it, rounded to integers, clipped to [w, n], with the rounding
  remainder given to the lowest layers so that the layers' mean is the mean
  budget; every head of a layer shares the layer's budget;
* adaptive: inside each layer the H heads share H (c - w) selected tokens,
  taken as the highest pooled SnapKV scores over all heads of the layer
  (ties to the lower head, then the lower position); head h keeps w plus the
  number of its tokens taken;
* token-based H2O: a prefix token's score is the attention it receives,
  accumulated over every prompt position (Sec. 2: heavy hitters by
  accumulated attention scores).  Reading: every query head of the KV head's
  group and every prompt position i (the window included) contribute their
  causal attention row softmax(q_i K^T / sqrt(d)) over keys 0..i; the score of
  prefix token j is the sum of those rows' entries at j.  The retained set is
  the top c - w prefix tokens by that score with no pooling (pool width 1)
  plus the w most recent tokens, and the merge is GRKV's value step on the
  window queries, as for any front-end.

Parity status: pinned by ``tests/test_oracle_frontend.py`` (uniform budgets
reduce to the batched oracle, brute-force joint top-k, closed forms of the
schedule; the accumulated attention by brute force, its zero-query closed
form in harmonic numbers, row normalisation and a dominant key).
"""
from __future__ import annotations

import numpy as np

from . import grkv_oracle as V

__all__ = ["pyramid_budgets", "adaptive_budgets", "compress_ragged", "packed_offsets",
           "h2o_scores", "compress_h2o"]


def pyramid_budgets(layers: int, kv_heads: int, mean_budget: int, window: int, n: int,
                    ratio: float = 0.5) -> np.ndarray:
    """Per-unit budgets [layers * kv_heads] of the pyramid schedule."""
    L = int(layers)
    if L == 1:
        per = np.array([mean_budget], dtype=np.int64)
    else:
        top = ratio * mean_budget
        bot = (2.0 - ratio) * mean_budget
        raw = bot + (top - bot) * np.arange(L) / (L - 1)
        per = np.floor(raw + 0.5).astype(np.int64)
        per = np.clip(per, window, n)
        # rounding remainder to the lowest layers, one token each, keeping [w, n]
        diff = L * mean_budget - int(per.sum())
        l = 0
        while diff != 0 and l < 4 * L:
            j = l % L
            step = 1 if diff > 0 else -1
            if window <= per[j] + step <= n:
                per[j] += step
                diff -= step
            l += 1
    return np.repeat(per, kv_heads)


def adaptive_budgets(pooled: np.ndarray, layers: int, kv_heads: int, budget: int,
                     window: int) -> np.ndarray:
    """Per-unit budgets from the pooled scores [U, P] (U = layers * kv_heads,
    units of a layer adjacent): a joint top-(H (c - w)) per layer."""
    U, P = pooled.shape
    H = int(kv_heads)
    out = np.empty(U, dtype=np.int64)
    for l in range(layers):
        p = np.asarray(pooled[l * H:(l + 1) * H], dtype=np.float64)
        k = min(H * (budget - window), H * P)
        head = np.repeat(np.arange(H), P)
        pos = np.tile(np.arange(P), H)
        order = np.lexsort((pos, head, -p.ravel()))
        taken = np.bincount(head[order[:k]], minlength=H)
        out[l * H:(l + 1) * H] = window + taken
    return out


def packed_offsets(budgets) -> np.ndarray:
    """Start of each unit's retained slots in the packed outputs."""
    b = np.asarray(budgets, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(b)[:-1]]) if b.size else b


def compress_ragged(q_obs, K, Vv, budgets, window, pool_kernel, lam, opt=None, units=None):
    """Every unit compressed with its own budget (float64 values in).  Returns
    the per-unit ``compress_unit`` results."""
    U = K.shape[0]
    units = range(U) if units is None else units
    return [V.compress_unit(q_obs[u], K[u], Vv[u], window, int(budgets[u]), pool_kernel, lam, opt)
            for u in units]


def h2o_scores(q_all, K, window, all_columns=False):
    """Accumulated attention (H2O's heavy-hitter score) of one unit.

    q_all [G, n, d]: the queries of every prompt position for the G query
    heads of the KV head; K [n, d].  Row (g, i) is the causal attention of
    position i, softmax over keys 0..i of q_{g,i} . k_j / sqrt(d); the score
    of token j is the sum over all rows of their entries at j.  Returns the
    prefix scores [n - w] (all n columns with ``all_columns``)."""
    q_all = np.asarray(q_all, dtype=np.float64)
    G, n, d = q_all.shape
    Kd = np.asarray(K, dtype=np.float64)
    j = np.arange(n)
    s = np.zeros(n, dtype=np.float64)
    for g in range(G):
        L = (q_all[g] @ Kd.T) / np.sqrt(d)
        L = np.where(j[None, :] <= j[:, None], L, -np.inf)   # row i sees keys 0..i
        A, _ = V.softmax_rows(L)
        s += A.sum(axis=0)
    return s if all_columns else s[: n - window]


def compress_h2o(q_all, q_obs, K, Vv, window, budget, lam, opt=None):
    """H2O retention (accumulated-attention scores, no pooling) followed by
    GRKV's value step on the window queries q_obs [G, w, d]."""
    s = h2o_scores(q_all, K, window)
    return V.compress_unit(q_obs, K, Vv, window, budget, 1, lam, opt=opt, scores=s)
