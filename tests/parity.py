"""Shared helpers for GPU-vs-oracle parity tests.

The GPU path is called through its C ABI (via the package binding); the
oracle is the plain float64 implementation in ``oracle/``.  Both take their
inputs from ``workloads`` with the same seeds.
"""
from __future__ import annotations

import numpy as np

import workloads as W
from oracle import grkv_oracle as O

# parity tolerances: merged values and the post-merge discrepancy (relative)
V_TOL = 2e-3
D_TOL = 2e-3


def to_device(arr, dtype):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def run_gpu(cfg, q, K, V, **opts):
    import torch
    import paper_2605_31105_amd as G
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    res = G.compress(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam, **opts)
    torch.cuda.synchronize()
    inter = {k: v.cpu().numpy() for k, v in G.intermediates(res).items()}
    out = dict(idx=res.idx.cpu().numpy(), v_out=res.v_out.cpu().numpy(),
               stats=res.stats.cpu().numpy(), **inter)
    kc = res.k_out.cpu()
    out["k_out"] = kc.view(torch.int16).numpy().view(np.uint16) if cfg.dtype == "bf16" else kc.numpy()
    return out


def oracle_unit(cfg, q, K, V, u, opt=None, idx=None, scores=None):
    qd, Kd, Vd = (W.decode(a[u], cfg.dtype) for a in (q, K, V))
    return O.compress_unit(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam,
                           opt=opt, idx=idx, scores=scores)


def check_unit(cfg, q, K, V, gpu, u, slot=None, opt=None, report=None, scores=None):
    """Compare GPU outputs of unit ``u`` (row ``slot`` of the GPU batch) with
    the oracle (selection from ``scores`` when given).  Returns a dict of error
    figures; asserts the parity bar."""
    slot = u if slot is None else slot
    r = oracle_unit(cfg, q, K, V, u, opt=opt, scores=scores)
    idx_g = gpu["idx"][slot].astype(np.int64)
    diff = np.setdiff1d(r["idx"], idx_g).size
    info = {"unit": u, "idx_mismatch": int(diff)}
    # retained indices: exact, ties to the lower position
    assert diff == 0 and np.array_equal(idx_g, r["idx"]), \
        "unit %d: %d retained positions differ" % (u, diff)
    # K0: bit-exact copy of the input rows
    assert np.array_equal(gpu["k_out"][slot], K[u][idx_g])
    # fixed set: exact
    assert np.array_equal(gpu["fixed"][slot].astype(bool), r["fixed"])
    # merged values
    vmax = np.abs(r["Vstar"]).max()
    v_err = np.abs(gpu["v_out"][slot] - r["Vstar"]).max() / vmax
    info["v_err"] = float(v_err)
    assert v_err <= V_TOL, "unit %d: v_out rel err %.3e" % (u, v_err)
    # discrepancy: reported by the kernel, and re-evaluated in fp64 on the GPU output
    st = gpu["stats"][slot]
    assert st[3] == r["status"]
    d_rep = abs(st[2] - r["D_after"]) / max(r["D_after"], 1e-30)
    d_eval = abs(O.discrepancy(r["Y"], r["X"], gpu["v_out"][slot].astype(np.float64))
                 - r["D_after"]) / max(r["D_after"], 1e-30)
    d_before = abs(st[1] - r["D_before"]) / max(r["D_before"], 1e-30)
    y2_err = abs(st[0] - r["y2"]) / max(r["y2"], 1e-30)
    info.update(d_rep=float(d_rep), d_eval=float(d_eval), d_before=float(d_before),
                y2_err=float(y2_err))
    # stats[0] = ||Y||^2 and stats[1] = D_before (Eq. 4 at V0), same relative bar as D_after
    assert y2_err <= D_TOL, "unit %d: ||Y||^2 rel err %.3e" % (u, y2_err)
    if r["D_before"] > 1e-12:
        assert d_before <= D_TOL, "unit %d: D_before rel err %.3e" % (u, d_before)
    else:
        assert st[1] <= 1e-6, "unit %d: D_before %.3e where the oracle has %.3e" % (u, st[1], r["D_before"])
    if r["D_after"] > 1e-12:
        assert d_rep <= D_TOL and d_eval <= D_TOL, "unit %d: D errs %.3e %.3e" % (u, d_rep, d_eval)
    else:
        assert st[2] <= 1e-6 and O.discrepancy(r["Y"], r["X"], gpu["v_out"][slot].astype(np.float64)) <= 1e-6
    # intermediates
    info["lse_err"] = float(np.abs(gpu["lse"][slot] - r["lse"]).max())
    info["y_err"] = float(np.abs(gpu["y"][slot] - r["Y"]).max() / max(np.abs(r["Y"]).max(), 1e-30))
    if K.shape[1] > cfg.window:
        info["p_err"] = float(np.abs(gpu["pooled"][slot] - r["p"]).max() / r["p"].max())
    assert info["lse_err"] < 1e-4 and info["y_err"] < 1e-3, info
    if report is not None:
        report.append(info)
    return info
