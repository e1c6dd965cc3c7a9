"""MI355X (gfx950) GRKV prefill-compression path: Python binding.

Argument marshalling only.  Every step of the computation runs in the HIP
kernels of ``libgrkv.so`` behind the C ABI declared in ``include/grkv.h``;
PyTorch supplies device memory and the stream.  Importing works without a GPU;
calling ``compress`` requires the built library and a ROCm device, and raises
if either is missing (there is no CPU fallback).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

__all__ = [
    "GRKV_OK", "GRKV_ERR_INVALID", "GRKV_ERR_WORKSPACE", "GRKV_ERR_UNSUPPORTED",
    "GRKV_ERR_HIP", "GrkvError", "lib", "lib_path", "Problem", "Options", "Outputs",
    "Layout", "workspace_bytes", "workspace_layout", "compress", "Result",
    "intermediates", "EXPORTED_SYMBOLS", "KeyOptions", "workspace_bytes_kv", "compress_kv",
    "KEY_CONVERGED", "KEY_MAX_ITER", "KEY_SKIPPED", "KEY_BREAKDOWN", "carrier_stats",
    "CARRIER_METRICS", "compress_ragged", "pyramid_budgets", "adaptive_budgets",
    "workspace_bytes_ragged", "compress_noalloc", "NOALLOC_SCRATCH_BYTES", "h2o_scores",
    "compress_scored", "h2o_workspace_bytes",
]

GRKV_OK, GRKV_ERR_INVALID, GRKV_ERR_WORKSPACE, GRKV_ERR_UNSUPPORTED, GRKV_ERR_HIP = 0, -1, -2, -3, -4
GRKV_BF16, GRKV_F32 = 0, 1
STAGES = ("full_lse", "full_lse_combine", "full_prob", "full_y", "select", "gather",
          "ret_lse", "ret_lse_combine", "ret_prob", "resid", "gram", "solve", "update", "key")
NUM_STAGES = len(STAGES)
EXPORTED_SYMBOLS = ("grkv_compress", "grkv_workspace_bytes", "grkv_workspace_layout",
                    "grkv_default_options", "grkv_status_string", "grkv_compress_kv",
                    "grkv_workspace_bytes_kv", "grkv_default_key_options", "grkv_carrier_stats",
                    "grkv_compress_ragged", "grkv_workspace_bytes_ragged", "grkv_pyramid_budgets",
                    "grkv_adaptive_budgets", "grkv_compress_noalloc", "grkv_h2o_scores",
                    "grkv_h2o_workspace_bytes", "grkv_compress_scored")
NOALLOC_SCRATCH_BYTES = 64 << 20
KEY_CONVERGED, KEY_MAX_ITER, KEY_SKIPPED, KEY_BREAKDOWN = 1, 2, 3, 4
CARRIER_METRICS = ("b", "b_eff", "a_max", "gini", "boundary_fraction", "boundary_share",
                   "enrichment", "boundary_interior_load")

_PKG = os.path.dirname(os.path.abspath(__file__))


def lib_path() -> str:
    return os.path.join(_PKG, "libgrkv.so")


class GrkvError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("grkv status %d: %s" % (status, msg))
        self.status = status


class Problem(ctypes.Structure):
    _fields_ = [("units", ctypes.c_int32), ("group", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Options(ctypes.Structure):
    _fields_ = [("n_sink", ctypes.c_int32), ("beta", ctypes.c_float),
                ("fix_window", ctypes.c_int32), ("causal_window", ctypes.c_int32)]


class Outputs(ctypes.Structure):
    _fields_ = [("idx", ctypes.c_void_p), ("k_out", ctypes.c_void_p),
                ("v_out", ctypes.c_void_p), ("stats", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
                ("stage_events", ctypes.POINTER(ctypes.c_void_p))]


class KeyOptions(ctypes.Structure):
    _fields_ = [("lambda_k", ctypes.c_float), ("max_iter", ctypes.c_int32), ("tol", ctypes.c_float),
                ("steps", ctypes.c_int32)]


class Layout(ctypes.Structure):
    _fields_ = [(f, ctypes.c_size_t) for f in
                ("lse", "y", "score", "pooled", "fixed", "resid", "gram", "z", "total")]


_LIB = None


def lib() -> ctypes.CDLL:
    """Load libgrkv.so (once).  Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError("libgrkv.so is not built: run `python -m paper_2605_31105_amd.build`")
        L = ctypes.CDLL(path)
        P = ctypes.POINTER
        L.grkv_compress.restype = ctypes.c_int
        L.grkv_compress.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
                                    P(Problem), P(Options), P(Outputs)]
        L.grkv_compress_noalloc.restype = ctypes.c_int
        L.grkv_compress_noalloc.argtypes = L.grkv_compress.argtypes
        L.grkv_compress_scored.restype = ctypes.c_int
        L.grkv_compress_scored.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
                                           P(Problem), P(Options), ctypes.c_void_p, P(Outputs)]
        L.grkv_h2o_scores.restype = ctypes.c_int
        L.grkv_h2o_scores.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int32, ctypes.c_void_p, P(Problem), ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_size_t]
        L.grkv_h2o_workspace_bytes.restype = ctypes.c_size_t
        L.grkv_h2o_workspace_bytes.argtypes = [P(Problem), ctypes.c_int64]
        L.grkv_workspace_bytes.restype = ctypes.c_size_t
        L.grkv_workspace_bytes.argtypes = [P(Problem), ctypes.c_int64, ctypes.c_int32, ctypes.c_int32]
        L.grkv_workspace_layout.restype = ctypes.c_int
        L.grkv_workspace_layout.argtypes = [P(Problem), ctypes.c_int64, ctypes.c_int32,
                                            ctypes.c_int32, P(Layout)]
        L.grkv_default_options.restype = None
        L.grkv_default_options.argtypes = [P(Options)]
        L.grkv_compress_kv.restype = ctypes.c_int
        L.grkv_compress_kv.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
                                       P(Problem), P(Options), P(Outputs), P(KeyOptions),
                                       ctypes.c_void_p, ctypes.c_void_p]
        L.grkv_workspace_bytes_kv.restype = ctypes.c_size_t
        L.grkv_workspace_bytes_kv.argtypes = [P(Problem), ctypes.c_int64, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.c_int32]
        L.grkv_default_key_options.restype = None
        L.grkv_default_key_options.argtypes = [P(KeyOptions), ctypes.c_float]
        L.grkv_carrier_stats.restype = ctypes.c_int
        L.grkv_carrier_stats.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                         P(Problem), ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p]
        L.grkv_compress_ragged.restype = ctypes.c_int
        L.grkv_compress_ragged.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
                                           P(Problem), P(Options), P(Outputs)]
        L.grkv_workspace_bytes_ragged.restype = ctypes.c_size_t
        L.grkv_workspace_bytes_ragged.argtypes = [P(Problem), ctypes.c_int64, ctypes.c_int32,
                                                  ctypes.c_void_p]
        L.grkv_pyramid_budgets.restype = ctypes.c_int
        L.grkv_pyramid_budgets.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                           ctypes.c_void_p]
        L.grkv_adaptive_budgets.restype = ctypes.c_int
        L.grkv_adaptive_budgets.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_void_p]
        L.grkv_status_string.restype = ctypes.c_char_p
        L.grkv_status_string.argtypes = [ctypes.c_int]
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().grkv_status_string(status).decode()


def _check(status: int):
    if status != GRKV_OK:
        raise GrkvError(status, status_string(status))


def workspace_bytes(units, group, head_dim, dtype, n, window, budget) -> int:
    prob = Problem(units, group, head_dim, dtype)
    return int(lib().grkv_workspace_bytes(ctypes.byref(prob), n, window, budget))


def workspace_layout(units, group, head_dim, dtype, n, window, budget) -> Layout:
    prob = Problem(units, group, head_dim, dtype)
    lay = Layout()
    _check(lib().grkv_workspace_layout(ctypes.byref(prob), n, window, budget, ctypes.byref(lay)))
    return lay


def workspace_bytes_kv(units, group, head_dim, dtype, n, window, budget, steps=1) -> int:
    prob = Problem(units, group, head_dim, dtype)
    return int(lib().grkv_workspace_bytes_kv(ctypes.byref(prob), n, window, budget, steps))


def workspace_bytes_ragged(units, group, head_dim, dtype, n, window, budgets) -> int:
    import numpy as np
    prob = Problem(units, group, head_dim, dtype)
    b = np.ascontiguousarray(np.asarray(budgets, dtype=np.int32))
    return int(lib().grkv_workspace_bytes_ragged(ctypes.byref(prob), n, window,
                                                 b.ctypes.data_as(ctypes.c_void_p)))


@dataclass
class Result:
    idx: "object"        # int32 [U, c]
    k_out: "object"      # input dtype [U, c, d]
    v_out: "object"      # float32 [U, c, d]
    stats: "object"      # float32 [U, 4]
    workspace: "object"  # uint8 workspace, see intermediates()
    shape: tuple         # (U, G, d, dtype, n, window, budget)


def _prepare(q_obs, K, V, window, budget, need_fn, n_sink, beta, fix_window, causal_window,
             stream, workspace, out, stage_events):
    import torch

    if not (q_obs.is_cuda and K.is_cuda and V.is_cuda):
        raise ValueError("q_obs, K and V must be device tensors")
    if not (q_obs.dtype == K.dtype == V.dtype) or K.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("q_obs, K, V must share dtype bfloat16 or float32")
    if not (q_obs.is_contiguous() and K.is_contiguous() and V.is_contiguous()):
        raise ValueError("inputs must be contiguous")
    U, G, w, d = q_obs.shape
    if w != window or K.shape[0] != U or K.shape[2] != d or V.shape != K.shape:
        raise ValueError("shape mismatch: q_obs %s K %s V %s window %d"
                         % (tuple(q_obs.shape), tuple(K.shape), tuple(V.shape), window))
    n = K.shape[1]
    dt = GRKV_BF16 if K.dtype == torch.bfloat16 else GRKV_F32
    dev = K.device
    need = need_fn(U, G, d, dt, n, window, budget)
    if need == 0:
        # let the library report the precise error
        need = 256
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if out is None:
        out = Result(idx=torch.empty((U, budget), dtype=torch.int32, device=dev),
                     k_out=torch.empty((U, budget, d), dtype=K.dtype, device=dev),
                     v_out=torch.empty((U, budget, d), dtype=torch.float32, device=dev),
                     stats=torch.empty((U, 4), dtype=torch.float32, device=dev),
                     workspace=workspace, shape=())
    out.workspace = workspace
    out.shape = (U, G, d, dt, n, window, budget)
    prob = Problem(U, G, d, dt)
    opt = Options(n_sink, beta, 1 if fix_window else 0, 1 if causal_window else 0)
    outs = Outputs(out.idx.data_ptr(), out.k_out.data_ptr(), out.v_out.data_ptr(),
                   out.stats.data_ptr(), workspace.data_ptr(), workspace.numel(),
                   stage_events)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    return out, prob, opt, outs, handle, n


def compress(q_obs, K, V, window: int, budget: int, pool_kernel: int, lam: float, *,
             n_sink: int = 4, beta: float = 0.10, fix_window: bool = True,
             causal_window: bool = True, stream=None, workspace=None, out=None,
             stage_events=None) -> Result:
    """GRKV compression of U units on the GPU.

    q_obs [U, G, w, d], K and V [U, n, d]: contiguous CUDA tensors of one dtype
    (bfloat16 or float32).  Returns the retained indices, K0, the merged V*,
    per-unit stats {||Y||^2, D_before, D_after, status} and the workspace.
    ``workspace`` (uint8, >= workspace_bytes) and ``out`` (a Result whose
    tensors are reused) avoid allocations in timed loops.  ``stage_events`` is
    an optional ctypes array of 2 * NUM_STAGES event handles (see grkv.h).
    """
    out, prob, opt, outs, handle, n = _prepare(
        q_obs, K, V, window, budget, workspace_bytes, n_sink, beta, fix_window, causal_window,
        stream, workspace, out, stage_events)
    st = lib().grkv_compress(q_obs.data_ptr(), K.data_ptr(), V.data_ptr(), n, window, budget,
                             pool_kernel, float(lam), ctypes.c_void_p(handle),
                             ctypes.byref(prob), ctypes.byref(opt), ctypes.byref(outs))
    _check(st)
    return out


def compress_noalloc(q_obs, K, V, window: int, budget: int, pool_kernel: int, lam: float, *,
                     out: Result, n_sink: int = 4, beta: float = 0.10, fix_window: bool = True,
                     causal_window: bool = True, stream=None) -> Result:
    """``compress`` through the entry point that allocates nothing: the
    library's own per-device scratch array (NOALLOC_SCRATCH_BYTES) serves as the
    workspace.  ``out`` (a Result with idx, k_out, v_out and stats of the
    right shapes) is required, so this call allocates no device memory either.
    Calls that overlap on one device race on the shared scratch array."""
    import torch

    if not (q_obs.is_cuda and K.is_cuda and V.is_cuda):
        raise ValueError("q_obs, K and V must be device tensors")
    if not (q_obs.dtype == K.dtype == V.dtype) or K.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("q_obs, K, V must share dtype bfloat16 or float32")
    if not (q_obs.is_contiguous() and K.is_contiguous() and V.is_contiguous()):
        raise ValueError("inputs must be contiguous")
    U, G, w, d = q_obs.shape
    if w != window or K.shape[0] != U or K.shape[2] != d or V.shape != K.shape:
        raise ValueError("shape mismatch: q_obs %s K %s V %s window %d"
                         % (tuple(q_obs.shape), tuple(K.shape), tuple(V.shape), window))
    n = K.shape[1]
    if (tuple(out.idx.shape) != (U, budget) or tuple(out.k_out.shape) != (U, budget, d)
            or tuple(out.v_out.shape) != (U, budget, d) or tuple(out.stats.shape) != (U, 4)
            or out.k_out.dtype != K.dtype or out.v_out.dtype != torch.float32
            or out.idx.dtype != torch.int32 or out.stats.dtype != torch.float32):
        raise ValueError("out tensors do not match the call's shapes")
    dt = GRKV_BF16 if K.dtype == torch.bfloat16 else GRKV_F32
    prob = Problem(U, G, d, dt)
    opt = Options(n_sink, beta, 1 if fix_window else 0, 1 if causal_window else 0)
    outs = Outputs(out.idx.data_ptr(), out.k_out.data_ptr(), out.v_out.data_ptr(),
                   out.stats.data_ptr(), None, 0, None)
    if stream is None:
        stream = torch.cuda.current_stream(K.device)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    with torch.cuda.device(K.device):
        st = lib().grkv_compress_noalloc(q_obs.data_ptr(), K.data_ptr(), V.data_ptr(), n, window,
                                         budget, pool_kernel, float(lam), ctypes.c_void_p(handle),
                                         ctypes.byref(prob), ctypes.byref(opt), ctypes.byref(outs))
    _check(st)
    out.workspace = None
    out.shape = (U, G, d, dt, n, window, budget)
    return out


def h2o_workspace_bytes(units, group, head_dim, dtype, n) -> int:
    prob = Problem(units, group, head_dim, dtype)
    return int(lib().grkv_h2o_workspace_bytes(ctypes.byref(prob), n))


def h2o_scores(q_all, K, window: int, *, stream=None, workspace=None, out=None):
    """H2O accumulated-attention scores of every prefix token (grkv_h2o_scores).

    q_all [U, G, n, d] (the queries of every prompt position) and K [U, n, d]:
    contiguous bfloat16 device tensors.  Returns float32 scores [U, n - window]."""
    import torch

    if not (q_all.is_cuda and K.is_cuda) or not (q_all.is_contiguous() and K.is_contiguous()):
        raise ValueError("q_all and K must be contiguous device tensors")
    if q_all.dtype != torch.bfloat16 or K.dtype != torch.bfloat16:
        raise ValueError("q_all and K must be bfloat16")
    U, Gq, n, d = q_all.shape
    if tuple(K.shape) != (U, n, d):
        raise ValueError("shape mismatch: q_all %s K %s" % (tuple(q_all.shape), tuple(K.shape)))
    need = max(256, h2o_workspace_bytes(U, Gq, d, GRKV_BF16, n))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=K.device)
    if out is None:
        out = torch.empty((U, max(n - window, 0)), dtype=torch.float32, device=K.device)
    prob = Problem(U, Gq, d, GRKV_BF16)
    if stream is None:
        stream = torch.cuda.current_stream(K.device)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    _check(lib().grkv_h2o_scores(q_all.data_ptr(), K.data_ptr(), n, window,
                                 ctypes.c_void_p(handle), ctypes.byref(prob),
                                 out.data_ptr() if out.numel() else None, workspace.data_ptr(),
                                 workspace.numel()))
    return out


def compress_scored(q_obs, K, V, window: int, budget: int, pool_kernel: int, lam: float,
                    scores, *, n_sink: int = 4, beta: float = 0.10, fix_window: bool = True,
                    causal_window: bool = True, stream=None, workspace=None, out=None,
                    stage_events=None) -> Result:
    """``compress`` with the selection ranking caller-supplied per-token scores
    (float32 [U, n - window], finite and non-negative) pooled with pool_kernel,
    instead of the window attention's column sums (grkv_compress_scored)."""
    import torch

    out, prob, opt, outs, handle, n = _prepare(
        q_obs, K, V, window, budget, workspace_bytes, n_sink, beta, fix_window, causal_window,
        stream, workspace, out, stage_events)
    if not (scores.is_cuda and scores.dtype == torch.float32 and scores.is_contiguous()):
        raise ValueError("scores must be a contiguous float32 device tensor")
    if tuple(scores.shape) != (K.shape[0], n - window):
        raise ValueError("scores must be [U, n - window]")
    st = lib().grkv_compress_scored(q_obs.data_ptr(), K.data_ptr(), V.data_ptr(), n, window,
                                    budget, pool_kernel, float(lam), ctypes.c_void_p(handle),
                                    ctypes.byref(prob), ctypes.byref(opt),
                                    scores.data_ptr() if scores.numel() else None,
                                    ctypes.byref(outs))
    _check(st)
    return out


def compress_kv(q_obs, K, V, window: int, budget: int, pool_kernel: int, lam: float, *,
                lambda_k=None, max_iter: int = 64, tol: float = 1e-5, steps: int = 1,
                n_sink: int = 4,
                beta: float = 0.10, fix_window: bool = True, causal_window: bool = True,
                stream=None, workspace=None, out=None, k_star=None, cg_info=None,
                stage_events=None):
    """``compress`` followed by the key step (bfloat16 inputs, G*w <= 128), and
    for ``steps`` > 1 further alternating value and key steps.

    Returns ``(result, k_star, cg_info)``: k_star float32 [U, c, d] holds the
    merged keys K*, cg_info float32 [U, 4] holds {CG iterations, final
    relative residual, KEY_* outcome, ||rhs||} of the last key step.
    ``lambda_k`` defaults to ``lam``."""
    import torch

    out, prob, opt, outs, handle, n = _prepare(
        q_obs, K, V, window, budget,
        lambda *a: workspace_bytes_kv(*a, steps=steps), n_sink, beta, fix_window,
        causal_window, stream, workspace, out, stage_events)
    U, d = q_obs.shape[0], q_obs.shape[3]
    if k_star is None:
        k_star = torch.empty((U, budget, d), dtype=torch.float32, device=K.device)
    if cg_info is None:
        cg_info = torch.empty((U, 4), dtype=torch.float32, device=K.device)
    kopt = KeyOptions(float(lam if lambda_k is None else lambda_k), int(max_iter), float(tol),
                      int(steps))
    st = lib().grkv_compress_kv(q_obs.data_ptr(), K.data_ptr(), V.data_ptr(), n, window, budget,
                                pool_kernel, float(lam), ctypes.c_void_p(handle),
                                ctypes.byref(prob), ctypes.byref(opt), ctypes.byref(outs),
                                ctypes.byref(kopt), ctypes.c_void_p(k_star.data_ptr()),
                                ctypes.c_void_p(cg_info.data_ptr()))
    _check(st)
    return out, k_star, cg_info


def carrier_stats(K, idx, group: int, stats=None, *, stream=None, assign=None, counts=None,
                  metrics=None, l_common=None):
    """Key-cosine carrier assignment and its load metrics (see grkv.h).

    K [U, n, d] bfloat16 device tensor, idx [U, c] int32 (from ``compress``),
    stats [U, 4] optional (gives L_common).  Returns ``(assign [U, n] int32,
    counts [U, c] int32, metrics [U, 8] float32, l_common [1] float32 or None)``;
    the metric columns are named in CARRIER_METRICS."""
    import torch

    if not (K.is_cuda and idx.is_cuda) or not K.is_contiguous() or not idx.is_contiguous():
        raise ValueError("K and idx must be contiguous device tensors")
    U, n, d = K.shape
    c = idx.shape[1]
    dt = GRKV_BF16 if K.dtype == torch.bfloat16 else GRKV_F32
    dev = K.device
    if assign is None:
        assign = torch.empty((U, n), dtype=torch.int32, device=dev)
    if counts is None:
        counts = torch.empty((U, c), dtype=torch.int32, device=dev)
    if metrics is None:
        metrics = torch.empty((U, 8), dtype=torch.float32, device=dev)
    if stats is not None and l_common is None:
        l_common = torch.empty(1, dtype=torch.float32, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    prob = Problem(U, group, d, dt)
    ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
    st = lib().grkv_carrier_stats(K.data_ptr(), n, c, ctypes.byref(prob), idx.data_ptr(),
                                  ptr(stats), ctypes.c_void_p(handle), assign.data_ptr(),
                                  ptr(counts), metrics.data_ptr(),
                                  ptr(l_common) if stats is not None else None)
    _check(st)
    return assign, counts, metrics, (l_common if stats is not None else None)


def pyramid_budgets(layers: int, kv_heads: int, mean_budget: int, window: int, n: int,
                    ratio: float = 0.5):
    """Per-unit budgets (numpy int32 [layers * kv_heads]) of the pyramid schedule."""
    import numpy as np
    out = np.empty(layers * kv_heads, dtype=np.int32)
    _check(lib().grkv_pyramid_budgets(layers, kv_heads, mean_budget, window, n, float(ratio),
                                      out.ctypes.data_as(ctypes.c_void_p)))
    return out


def adaptive_budgets(pooled, layers: int, kv_heads: int, budget: int, window: int, *,
                     stream=None, out=None):
    """Per-unit budgets (int32 device tensor [U]) from the pooled scores [U, n - w]
    of a ``compress`` call (see ``intermediates``)."""
    import torch

    if not pooled.is_cuda or pooled.dtype != torch.float32 or not pooled.is_contiguous():
        raise ValueError("pooled must be a contiguous float32 device tensor")
    U, P = pooled.shape
    n = P + window
    if out is None:
        out = torch.empty(U, dtype=torch.int32, device=pooled.device)
    if stream is None:
        stream = torch.cuda.current_stream(pooled.device)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    _check(lib().grkv_adaptive_budgets(ctypes.c_void_p(pooled.data_ptr()), layers, kv_heads, n,
                                       window, budget, ctypes.c_void_p(handle),
                                       ctypes.c_void_p(out.data_ptr())))
    return out


def compress_ragged(q_obs, K, V, window: int, budgets, pool_kernel: int, lam: float, *,
                    n_sink: int = 4, beta: float = 0.10, fix_window: bool = True,
                    causal_window: bool = True, stream=None, workspace=None, out=None,
                    stage_events=None):
    """Every unit compressed with its own budget (``budgets``: host sequence of U
    ints).  Returns ``(idx, k_out, v_out, stats, offsets)`` with the packed
    layout of grkv.h (unit u at slots offsets[u] .. offsets[u] + budgets[u]).
    ``out``: the first four of a previous call's results with the same budgets,
    reused as the outputs.  ``stage_events``: as for ``compress`` (recorded on
    the bf16 path, where one launch per stage serves every unit)."""
    import numpy as np
    import torch

    if not (q_obs.is_cuda and K.is_cuda and V.is_cuda):
        raise ValueError("q_obs, K and V must be device tensors")
    U, G, w, d = q_obs.shape
    n = K.shape[1]
    b = np.ascontiguousarray(np.asarray(budgets, dtype=np.int32))
    if b.shape != (U,) or w != window:
        raise ValueError("budgets must hold one budget per unit")
    dt = GRKV_BF16 if K.dtype == torch.bfloat16 else GRKV_F32
    prob = Problem(U, G, d, dt)
    need = int(lib().grkv_workspace_bytes_ragged(ctypes.byref(prob), n, window,
                                                 b.ctypes.data_as(ctypes.c_void_p)))
    dev = K.device
    if workspace is None or workspace.numel() < max(need, 256):
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    tot = int(b.sum())
    if out is not None:
        idx, k_out, v_out, stats = out[:4]
        if idx.numel() != tot or k_out.shape != (tot, d) or stats.shape != (U, 4):
            raise ValueError("out does not match the budgets")
    else:
        idx = torch.empty(tot, dtype=torch.int32, device=dev)
        k_out = torch.empty((tot, d), dtype=K.dtype, device=dev)
        v_out = torch.empty((tot, d), dtype=torch.float32, device=dev)
        stats = torch.empty((U, 4), dtype=torch.float32, device=dev)
    opt = Options(n_sink, beta, 1 if fix_window else 0, 1 if causal_window else 0)
    outs = Outputs(idx.data_ptr(), k_out.data_ptr(), v_out.data_ptr(), stats.data_ptr(),
                   workspace.data_ptr(), workspace.numel(), stage_events)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    _check(lib().grkv_compress_ragged(q_obs.data_ptr(), K.data_ptr(), V.data_ptr(), n, window,
                                      b.ctypes.data_as(ctypes.c_void_p), pool_kernel, float(lam),
                                      ctypes.c_void_p(handle), ctypes.byref(prob),
                                      ctypes.byref(opt), ctypes.byref(outs)))
    offsets = np.concatenate([[0], np.cumsum(b)[:-1]]).astype(np.int64)
    return idx, k_out, v_out, stats, offsets


def intermediates(res: Result) -> dict:
    """Views of the workspace intermediates of the last call (see grkv.h)."""
    import torch

    U, G, d, dt, n, w, c = res.shape
    lay = workspace_layout(U, G, d, dt, n, w, c)
    m = G * w
    mp = 32
    while mp < m:
        mp *= 2
    P = n - w
    ws = res.workspace

    def view(off, dtype, shape):
        count = 1
        for s in shape:
            count *= s
        nbytes = count * torch.empty((), dtype=dtype).element_size()
        return ws[off:off + nbytes].view(dtype).view(*shape)

    return {
        "lse": view(lay.lse, torch.float64, (U, mp))[:, :m],
        "y": view(lay.y, torch.float32, (U, mp, d))[:, :m],
        "score": view(lay.score, torch.float32, (U, P)),
        "pooled": view(lay.pooled, torch.float32, (U, P)),
        "fixed": view(lay.fixed, torch.uint8, (U, c)),
        "resid": view(lay.resid, torch.float32, (U, mp, d))[:, :m],
        "gram": view(lay.gram, torch.float32, (U, mp, mp))[:, :m, :m],
        "z": view(lay.z, torch.float32, (U, d, mp))[:, :, :m],
    }
