"""GPU parity of the H2O front-end: the accumulated-attention scores of every
prefix token against the float64 oracle, and compression driven by
caller-supplied scores (grkv_compress_scored) against the oracle's selection
and value step on the same scores."""
import numpy as np
import pytest

import workloads as W
from oracle import grkv_frontend_oracle as FO
from oracle import grkv_oracle as O
from tests.parity import check_unit, run_gpu, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SCORE_TOL = 1e-5   # per-element relative error of the fp32 scores


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _inputs(cfg):
    q, K, V = W.make_batch(cfg)
    q_all = W.make_prompt_queries(cfg, q, K)
    return q, K, V, q_all


def _gpu_scores(cfg, q_all, K):
    import paper_2605_31105_amd as G
    s = G.h2o_scores(to_device(q_all, cfg.dtype), to_device(K, cfg.dtype), cfg.window)
    torch.cuda.synchronize()
    return s.cpu().numpy()


SHAPES = [
    ("g4-d128", dict(layers=1, kv_heads=2, n=2048, budget=256)),
    ("g2-d64-ragged", dict(layers=1, kv_heads=2, group=2, head_dim=64, n=1000, budget=200)),
    ("g1", dict(layers=1, kv_heads=1, group=1, n=777, budget=100, window=8)),
    ("g8-w16", dict(layers=1, kv_heads=1, group=8, window=16, n=1500, budget=300)),
]


@pytest.mark.parametrize("label,over", SHAPES, ids=[s[0] for s in SHAPES])
def test_h2o_scores_match_oracle(label, over):
    cfg = W.config(2, **over)
    print("case h2o scores", label, flush=True)
    q, K, V, q_all = _inputs(cfg)
    got = _gpu_scores(cfg, q_all, K)
    for u in range(cfg.units):
        want = FO.h2o_scores(W.decode(q_all[u], cfg.dtype), W.decode(K[u], cfg.dtype), cfg.window)
        err = np.abs(got[u] - want) / want
        print(label, "unit", u, "max rel err %.2e" % err.max(), flush=True)
        assert err.max() <= SCORE_TOL


def test_h2o_scores_zero_queries_closed_form():
    # zero queries: s_j = G (H_n - H_j) (harmonic numbers)
    cfg = W.config(2, layers=1, kv_heads=1, n=3000, budget=256)
    q, K, V, q_all = _inputs(cfg)
    q_all[:] = 0
    got = _gpu_scores(cfg, q_all, K)[0]
    n, P = cfg.n, cfg.n - cfg.window
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, n + 1))])
    want = cfg.group * (H[n] - H[:P])
    assert np.max(np.abs(got - want) / want) <= SCORE_TOL


def test_compress_scored_matches_oracle_on_the_same_scores():
    # the GPU's fp32 scores given to both sides: selection exact, merge in tolerance
    import paper_2605_31105_amd as G
    cfg = W.config(2, layers=1, kv_heads=2, n=2048, budget=256, pool_kernel=1)
    q, K, V, q_all = _inputs(cfg)
    s = _gpu_scores(cfg, q_all, K)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    res = G.compress_scored(qd, Kd, Vd, cfg.window, cfg.budget, 1, cfg.lam,
                            torch.from_numpy(s).cuda())
    torch.cuda.synchronize()
    gpu = dict(idx=res.idx.cpu().numpy(), v_out=res.v_out.cpu().numpy(),
               stats=res.stats.cpu().numpy(),
               **{k: v.cpu().numpy() for k, v in G.intermediates(res).items()})
    gpu["k_out"] = res.k_out.cpu().view(torch.int16).numpy().view(np.uint16)
    for u in range(cfg.units):
        print(check_unit(cfg, q, K, V, gpu, u, scores=s[u].astype(np.float64)), flush=True)


@pytest.mark.parametrize("pool", [1, 7])
def test_h2o_end_to_end_against_oracle(pool):
    # H2O retention (GPU scores, GPU compression) against the oracle's own
    # fp64 scores and compression
    import paper_2605_31105_amd as G
    cfg = W.config(2, layers=1, kv_heads=2, n=2048, budget=256, pool_kernel=pool)
    q, K, V, q_all = _inputs(cfg)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    s = G.h2o_scores(to_device(q_all, cfg.dtype), Kd, cfg.window)
    res = G.compress_scored(qd, Kd, Vd, cfg.window, cfg.budget, pool, cfg.lam, s)
    torch.cuda.synchronize()
    for u in range(cfg.units):
        qo, Ko, Vo, qa = (W.decode(a[u], cfg.dtype) for a in (q, K, V, q_all))
        so = FO.h2o_scores(qa, Ko, cfg.window)
        r = O.compress_unit(qo, Ko, Vo, cfg.window, cfg.budget, pool, cfg.lam, scores=so)
        assert np.array_equal(res.idx[u].cpu().numpy(), r["idx"])
        v_err = np.abs(res.v_out[u].cpu().numpy() - r["Vstar"]).max() / np.abs(r["Vstar"]).max()
        print("pool", pool, "unit", u, "v_err %.2e" % v_err, flush=True)
        assert v_err <= 2e-3


def test_compress_scored_long_prefix_sample_misses_the_top():
    # a prefix past 32768 positions takes the long-prefix selection, whose
    # first brackets come from every 5th score (stride = ceil(P / 8192)); here
    # every sampled position holds a low score and the top-k lies among the
    # others, so the brackets fail their exact count check and both searches
    # run from the full range: the selection must still equal the oracle's
    import paper_2605_31105_amd as G
    cfg = W.config(2, layers=1, kv_heads=2, n=40000, budget=2048, pool_kernel=1)
    q, K, V = W.make_batch(cfg)
    P = cfg.n - cfg.window
    stride = -(-P // 8192)
    assert stride == 5
    rng = np.random.default_rng(11)
    s = (1.0 + rng.random((cfg.units, P))).astype(np.float32)
    s[:, ::stride] = (1e-3 * (1.0 + rng.random((cfg.units, (P + stride - 1) // stride)))).astype(np.float32)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    print("case scored long prefix, sampled positions low", flush=True)
    res = G.compress_scored(qd, Kd, Vd, cfg.window, cfg.budget, 1, cfg.lam,
                            torch.from_numpy(s).cuda())
    torch.cuda.synchronize()
    gpu = dict(idx=res.idx.cpu().numpy(), v_out=res.v_out.cpu().numpy(),
               stats=res.stats.cpu().numpy(),
               **{k: v.cpu().numpy() for k, v in G.intermediates(res).items()})
    gpu["k_out"] = res.k_out.cpu().view(torch.int16).numpy().view(np.uint16)
    for u in range(cfg.units):
        kept = gpu["idx"][u][: cfg.budget - cfg.window]
        assert np.all(kept % stride != 0)   # no sampled (low) position is kept
        print(check_unit(cfg, q, K, V, gpu, u, scores=s[u].astype(np.float64)), flush=True)
