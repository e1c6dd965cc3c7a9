"""Plain float64 CPU oracle of the carrier-concentration diagnostics.

TEST INFRASTRUCTURE ONLY, like the other oracle modules: imported by the test
suite, the smoke check and the benchmark's CPU-baseline leg, never by the
product path, and sharing no code with the HIP path.

The paper motivates GRKV by how a local merge rule loads the retained tokens
after span-based eviction (Sec. 1; App. A; App. B, "Quantitative Carrier
Concentration"): a key-similarity matcher, as in D2O/KVMerger, assigns every
evicted token to the retained token whose key has the highest cosine
similarity with its own, and the resulting loads a_i (evicted tokens assigned
to retained slot i) are summarised per unit by

* b = number of slots with a_i > 0 (active carriers),
* b_eff = (sum a)^2 / sum a^2 (effective carrier count),
* A_max = max a / (sum a / c) (maximum load over the mean load),
* the Gini coefficient of the loads,
* for span-based retention: boundary carriers (the first and the last retained
  token of every run of consecutive positions), their fraction of the slots,
  their share of the assignments, the enrichment (share / fraction) and the
  boundary / interior mean-load ratio (only when both kinds exist).

The paper also reports L_common, the window discrepancy summed over units:
sum ||Y_full - Y_comp||^2 / sum ||Y_full||^2.

Readings (the paper does not fix them): every retained token is a candidate
(no locality window); equal similarities go to the lower slot; a zero key has
cosine 0 with everything; the Gini coefficient is the mean absolute difference
over all ordered pairs divided by twice the mean.

Parity status: pinned by ``tests/test_oracle_carrier.py`` (brute force on tiny
inputs, scale invariance, closed forms of the metrics on constructed loads).
"""
from __future__ import annotations

import numpy as np

__all__ = ["cosine_matrix", "carrier_assignment", "carrier_metrics", "l_common"]


def cosine_matrix(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """cos(a_j, b_i) for rows of A against rows of B (0 where a norm is 0)."""
    na = np.linalg.norm(A, axis=1)
    nb = np.linalg.norm(B, axis=1)
    dots = A @ B.T
    den = na[:, None] * nb[None, :]
    return np.where(den > 0, dots / np.where(den > 0, den, 1.0), 0.0)


def carrier_assignment(K: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Slot (index into idx) of the retained token assigned to every token of
    the cache, or -1 for the retained tokens themselves: the highest key cosine
    similarity, ties to the lower slot."""
    n = K.shape[0]
    idx = np.asarray(idx, dtype=np.int64)
    retained = np.zeros(n, dtype=bool)
    retained[idx] = True
    ev = np.flatnonzero(~retained)
    out = np.full(n, -1, dtype=np.int64)
    if ev.size and idx.size:
        C = cosine_matrix(K[ev], K[idx])
        out[ev] = np.argmax(C, axis=1)   # first maximum = lowest slot
    return out


def _boundary_slots(idx: np.ndarray) -> np.ndarray:
    """True for the first and the last slot of each run of consecutive positions."""
    idx = np.asarray(idx, dtype=np.int64)
    c = idx.size
    first = np.ones(c, dtype=bool)
    last = np.ones(c, dtype=bool)
    if c > 1:
        first[1:] = idx[1:] != idx[:-1] + 1
        last[:-1] = idx[:-1] + 1 != idx[1:]
    return first | last


def carrier_metrics(assign: np.ndarray, idx: np.ndarray) -> dict:
    """The load summaries of App. B for one unit, from an assignment."""
    c = np.asarray(idx).size
    a = np.bincount(assign[assign >= 0], minlength=c).astype(np.float64)
    tot = a.sum()
    bnd = _boundary_slots(idx)
    out = dict(counts=a.astype(np.int64), b=float(np.count_nonzero(a)))
    if tot > 0:
        out["b_eff"] = tot * tot / float(np.sum(a * a))
        out["a_max"] = float(a.max()) / (tot / c)
        diff = np.abs(a[:, None] - a[None, :]).sum()
        out["gini"] = float(diff) / (2.0 * c * tot)
        frac = bnd.sum() / c
        ratio = a[bnd].sum() / tot
        out["boundary_fraction"] = float(frac)
        out["boundary_share"] = float(ratio)
        out["enrichment"] = float(ratio / frac)
        if bnd.any() and (~bnd).any():
            mi = a[~bnd].mean()
            out["boundary_interior_load"] = float(a[bnd].mean() / mi) if mi > 0 else float("inf")
        else:
            out["boundary_interior_load"] = float("nan")
    else:
        for k in ("b_eff", "a_max", "gini", "boundary_fraction", "boundary_share", "enrichment",
                  "boundary_interior_load"):
            out[k] = float("nan")
        out["boundary_fraction"] = float(bnd.sum() / c) if c else float("nan")
    return out


def l_common(y_full, y_comp) -> float:
    """sum ||Y_full - Y_comp||^2 / sum ||Y_full||^2 over all units given."""
    num = sum(float(np.sum((np.asarray(f) - np.asarray(g)) ** 2)) for f, g in zip(y_full, y_comp))
    den = sum(float(np.sum(np.asarray(f) ** 2)) for f in y_full)
    return num / den
