"""Plain float64 CPU oracle of GRKV's value-step prefill compression.

TEST INFRASTRUCTURE ONLY.  This file defines what the GPU path must compute;
it is written for a reader checking it against the paper, not for speed.  Only
the test suite, the smoke check and the benchmark's CPU-baseline leg may import
it.  It shares no code with the HIP path: no kernels, helpers or constants.

Per (layer, KV head) unit, following the paper's notation:

1. Window attention over the full cache (Sec. 3.1, standard attention;
   Sec. 3.2, window objective Eq. 4): the m = G*w window queries attend to all
   n cached keys, ``A = softmax(Q K^T / sqrt(d))``, ``Y = A V`` (the target of
   Algorithm 1's first step).
2. SnapKV-style span retention (Sec. 1 and Sec. 2 describe SnapKV as pooling the
   query-window attention scores over segments and keeping the top-k): column
   sums of ``A`` over the window rows, a box pooling of width k, and top-(c-w)
   selection over the prefix; the w window tokens are always kept.
3. Fixed tokens (Sec. 3.4 "Fixed tokens during optimization"; App. D.3): sink
   tokens, the window tokens and the top beta=10% retained tokens by score.
4. Value step (Eq. 6-8; Algorithm 1, value step; App. D.1):
   ``X = softmax(Q K_Ret^T / sqrt(d))``, ``R = Y - X V0``,
   ``Z = (X_G X_G^T + lambda I_m)^-1 R``, ``V*_G = V0_G + X_G^T Z``, ``V*_F = V0_F``.
   The primal form (Eq. 7 restricted to the free tokens) is computed too, as a
   cross-check of the dual.  Keys are kept: ``K* = K0``.

Readings of points the paper leaves open (all documented in the design notes):
grouped queries are stacked into m = G*w rows (row r = g*w + i, at position
n - w + i); the window rows are causally masked (row at position p sees keys
0..p) when ``causal_window`` is set; pooling is a zero-padded box sum of odd width
k, ranked as is (same order as an average pool); the budget c counts the w
window tokens; ties in the pooled score go to the lower position; the top-beta
fixed set is the first floor(beta*c) positions of the selection order; sinks are
the retained positions below ``n_sink`` (default 4) and are never forced in.

Parity status of every function here is pinned by the tests in
``tests/test_oracle_*.py`` (closed forms, brute force on tiny inputs,
least-squares and KKT checks, invariants).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "Options", "stack_queries", "query_positions", "window_logits",
    "softmax_rows", "selection_scores", "pool_box", "selection_order",
    "retained_index", "fixed_mask", "retained_attention", "merge_dual",
    "merge_primal", "discrepancy", "compress_unit", "merge_forced_unit",
    "compress", "STATUS_OK", "STATUS_SINGULAR",
]

STATUS_OK = 0
STATUS_SINGULAR = 1


class Options:
    """Knobs the paper fixes by default (Sec. 4.1 hyperparameters).

    n_sink: retained positions below this index are fixed (sink tokens).
    beta: fraction of the budget, taken from the top of the selection order,
          that stays fixed (paper default 10%).
    fix_window: the w observation-window tokens stay fixed (paper default).
    causal_window: window row at position p sees only keys 0..p.
    """

    def __init__(self, n_sink=4, beta=0.10, fix_window=True, causal_window=True):
        self.n_sink = int(n_sink)
        self.beta = float(np.float32(beta))   # the C ABI carries beta as float32
        self.fix_window = bool(fix_window)
        self.causal_window = bool(causal_window)


# ---------------------------------------------------------------- step 1 ----

def stack_queries(q_obs: np.ndarray) -> np.ndarray:
    """[G, w, d] window queries of one KV head -> [m, d] rows, r = g*w + i."""
    G, w, d = q_obs.shape
    return np.asarray(q_obs, dtype=np.float64).reshape(G * w, d)


def query_positions(G: int, w: int, n: int) -> np.ndarray:
    """Token position of each stacked row: the window is the last w prompt
    tokens (Sec. 3.2: the final query window is the surrogate), so row
    r = g*w + i sits at position n - w + i for every query head g."""
    return np.tile(np.arange(n - w, n, dtype=np.int64), G)


def window_logits(Q: np.ndarray, K: np.ndarray, pos: np.ndarray,
                  causal: bool) -> np.ndarray:
    """l[r, j] = q_r . k_j / sqrt(d) (Sec. 3.1), -inf where the causal rule hides
    key j from row r (j > pos[r])."""
    d = Q.shape[1]
    L = (Q @ K.T) / math.sqrt(d)
    if causal:
        j = np.arange(K.shape[0])
        L = np.where(j[None, :] <= pos[:, None], L, -np.inf)
    return L


def softmax_rows(L: np.ndarray):
    """Row softmax of logits with -inf entries; returns (A, lse)."""
    mx = np.max(L, axis=1, keepdims=True)
    e = np.exp(L - mx)
    z = e.sum(axis=1, keepdims=True)
    A = e / z
    lse = (mx + np.log(z))[:, 0]
    return A, lse


# ---------------------------------------------------------------- step 2 ----

def selection_scores(A: np.ndarray, prefix: int) -> np.ndarray:
    """SnapKV score of each prefix token: the attention it receives, summed over
    all window rows, s_j = sum_r A[r, j] for j < prefix = n - w."""
    return A[:, :prefix].sum(axis=0)


def pool_box(s: np.ndarray, k: int) -> np.ndarray:
    """1-D pooling over segments: p_j = sum_{t=j-h}^{j+h} s_t with h=(k-1)/2 and
    s_t = 0 outside the prefix.  Written as a direct window sum."""
    assert k >= 1 and k % 2 == 1
    h = (k - 1) // 2
    P = s.shape[0]
    p = np.zeros(P, dtype=np.float64)
    for j in range(P):
        lo, hi = max(0, j - h), min(P, j + h + 1)
        p[j] = s[lo:hi].sum()
    return p


def selection_order(p: np.ndarray) -> np.ndarray:
    """Prefix positions ordered by pooled score, highest first; equal scores go
    to the lower position first."""
    j = np.arange(p.shape[0])
    return np.lexsort((j, -p))


def retained_index(order: np.ndarray, n: int, w: int, budget: int) -> np.ndarray:
    """The c retained positions, ascending: the top c - w prefix positions of
    the selection order plus the whole window n-w..n-1."""
    sel = order[: budget - w]
    return np.sort(np.concatenate([sel, np.arange(n - w, n)])).astype(np.int64)


# ---------------------------------------------------------------- step 3 ----

def fixed_mask(idx: np.ndarray, order: np.ndarray, n: int, w: int, budget: int,
               opt: Options) -> np.ndarray:
    """Fixed set F over the retained slots (Sec. 3.4; App. D.3): sink tokens,
    the window tokens and the top floor(beta*c) selected tokens by score."""
    n_top = min(int(math.floor(opt.beta * budget)), budget - w)
    top = set(int(t) for t in order[:n_top])
    F = np.zeros(idx.shape[0], dtype=bool)
    for slot, pos in enumerate(idx):
        pos = int(pos)
        if pos < opt.n_sink:
            F[slot] = True
        if opt.fix_window and pos >= n - w:
            F[slot] = True
        if pos in top:
            F[slot] = True
    return F


# ---------------------------------------------------------------- step 4 ----

def retained_attention(Q, K0, idx, pos, causal):
    """X = softmax(Q K_Ret^T / sqrt(d)) over the retained keys (Algorithm 1,
    value step; App. D.1), with the same causal rule on retained positions."""
    d = Q.shape[1]
    L = (Q @ K0.T) / math.sqrt(d)
    if causal:
        L = np.where(idx[None, :] <= pos[:, None], L, -np.inf)
    X, _ = softmax_rows(L)
    return X


def merge_dual(X, Y, V0, F, lam):
    """Woodbury dual of the value step (Eq. 8; App. D.1 dual form; App. D.3 for
    fixed tokens).  Returns (dV, Z, R, status).

    R = Y - X_F V0_F - X_G V0_G = Y - X V0; N = X_G X_G^T + lam I_m;
    Z = N^-1 R; dV_G = X_G^T Z, dV_F = 0.  When N is not positive definite
    (only possible for lam = 0) the minimum-norm least-squares Z is used and the
    status is STATUS_SINGULAR."""
    m = X.shape[0]
    R = Y - X @ V0
    XG = np.where(F[None, :], 0.0, X)
    N = XG @ XG.T + lam * np.eye(m)
    status = STATUS_OK
    try:
        Lc = np.linalg.cholesky(N)
        Z = np.linalg.solve(Lc.T, np.linalg.solve(Lc, R))
    except np.linalg.LinAlgError:
        status = STATUS_SINGULAR
        Z = np.linalg.lstsq(N, R, rcond=None)[0]
    dV = XG.T @ Z
    return dV, Z, R, status


def merge_primal(X, Y, V0, F, lam):
    """Primal value step (Eq. 7) restricted to the free tokens G:
    (X_G^T X_G + lam I) dV_G = X_G^T (Y - X V0), dV_F = 0."""
    R = Y - X @ V0
    G = np.flatnonzero(~F)
    dV = np.zeros_like(V0)
    if G.size:
        XG = X[:, G]
        M = XG.T @ XG + lam * np.eye(G.size)
        dV[G] = np.linalg.solve(M, XG.T @ R)
    return dV


def discrepancy(Y, X, V):
    """Window objective (Eq. 4) normalised by the target energy, as in the
    paper's normalised common discrepancy: ||Y - X V||_F^2 / ||Y||_F^2 (the raw
    value when ||Y|| = 0)."""
    y2 = float(np.sum(Y * Y))
    e2 = float(np.sum((Y - X @ V) ** 2))
    return e2 / y2 if y2 > 0 else e2


# ------------------------------------------------------------- driver -------

def compress_unit(q_obs, K, V, window, budget, pool_kernel, lam, opt=None,
                  with_primal=False, idx=None, scores=None):
    """All steps for one unit on float64 inputs.

    q_obs [G, w, d], K [n, d], V [n, d] as exact float64 values.  When ``idx``
    is given the selection is skipped and that retained set is used (it must be
    ascending and end with the window).  When ``scores`` [n - w] is given, the
    selection ranks those per-token scores (pooled with the same box) instead
    of the window attention's column sums: the form a token-based eviction
    method such as H2O (Sec. 2) plugs in; the merge is unchanged.  Returns a
    dict with every intermediate, so tests can pin each step on its own."""
    opt = opt or Options()
    G, w, d = q_obs.shape
    n = K.shape[0]
    assert w == window and 1 <= w <= budget <= n
    Q = stack_queries(q_obs)
    pos = query_positions(G, w, n)
    L = window_logits(Q, K, pos, opt.causal_window)
    A, lse = softmax_rows(L)
    Y = A @ V
    prefix = n - w
    s = selection_scores(A, prefix) if scores is None else np.asarray(scores, dtype=np.float64)
    assert s.shape == (prefix,)
    p = pool_box(s, pool_kernel)
    order = selection_order(p)
    if idx is None:
        idx = retained_index(order, n, w, budget)
    idx = np.asarray(idx, dtype=np.int64)
    F = fixed_mask(idx, order, n, w, budget, opt)
    K0, V0 = K[idx], V[idx]
    X = retained_attention(Q, K0, idx, pos, opt.causal_window)
    dV, Z, R, status = merge_dual(X, Y, V0, F, lam)
    Vs = V0 + dV
    out = dict(Q=Q, pos=pos, L=L, A=A, lse=lse, Y=Y, s=s, p=p, order=order,
               idx=idx, fixed=F, K0=K0, V0=V0, X=X, R=R, Z=Z, dV=dV, Vstar=Vs,
               status=status, y2=float(np.sum(Y * Y)),
               D_before=discrepancy(Y, X, V0), D_after=discrepancy(Y, X, Vs))
    if with_primal:
        out["dV_primal"] = merge_primal(X, Y, V0, F, lam)
    return out


def merge_forced_unit(q_obs, K, V, idx, window, budget, pool_kernel, lam, opt=None):
    """Value step on a given retained set (used to check a GPU result whose
    retained set is taken as given)."""
    return compress_unit(q_obs, K, V, window, budget, pool_kernel, lam, opt, idx=idx)


def compress(q_obs, K, V, window, budget, pool_kernel, lam, opt=None, units=None):
    """Batched form over units with the C ABI's output shapes.

    q_obs [U, G, w, d], K/V [U, n, d] as float64 values.  Returns
    (idx [U, c] int64, k_out [U, c, d], v_out [U, c, d], stats [U, 4]) with
    stats = (||Y||^2, D_before, D_after, status)."""
    U = K.shape[0]
    units = range(U) if units is None else units
    idx_l, k_l, v_l, st_l = [], [], [], []
    for u in units:
        r = compress_unit(q_obs[u], K[u], V[u], window, budget, pool_kernel, lam, opt)
        idx_l.append(r["idx"])
        k_l.append(r["K0"])
        v_l.append(r["Vstar"])
        st_l.append([r["y2"], r["D_before"], r["D_after"], float(r["status"])])
    return np.stack(idx_l), np.stack(k_l), np.stack(v_l), np.array(st_l)
