"""Seeded synthetic inputs for the GRKV prefill-compression path.

This module only draws random numbers and rounds them to the storage type.
It holds none of the method's arithmetic (no attention, scoring, selection or
regression), so both the GPU path and the CPU oracle can take their inputs from
it without sharing any step of the computation.

The paper evaluates on LongBench and RULER with Llama-3.1-8B, Mistral-7B and
Qwen3-14B (Sec. 4.1).  None of those datasets or weights are used here; the
recipes below stand in for them with caches of the same shape (32 query heads
over 8 KV heads, head_dim 128, contexts of 8K-128K tokens, 10%-style budgets)
and a query window biased toward a few salient token spans, which is the
structure SnapKV-style span retention exploits (Sec. 1).

Per unit (one layer x one KV head) the generator draws, in this order:
channel scales -> outlier channels -> K -> V -> span count -> span slots ->
query noise, from ``numpy.random.default_rng(SeedSequence([cfg, layer, head]))``.
Each query row is ``0.5*eps + 1.5*mu`` where ``mu`` is the mean (in float64) of
the rounded key rows inside the salient spans and ``eps ~ N(0, I_d)``.

Storage: float32 configs keep float32 arrays; bfloat16 configs are held as
``uint16`` bit patterns produced by round-to-nearest-even from float32.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "Config", "CONFIGS", "config", "make_unit", "make_batch", "make_prompt_queries",
    "f32_to_bf16_bits", "bf16_bits_to_f32", "decode",
]


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload.  ``units = layers * kv_heads``."""
    cfg_id: int
    name: str
    layers: int
    kv_heads: int
    group: int          # query heads per KV head (GQA)
    head_dim: int
    n: int              # tokens in the full cache
    window: int         # observation-window length w
    budget: int         # retained tokens c (includes the w window tokens)
    pool_kernel: int
    lam: float
    dtype: str          # "f32" or "bf16"
    k_dist: str         # "normal", "scaled" (log-normal channel scales + outliers), "student_t3"
    span_count: tuple   # (lo, hi) inclusive; lo == hi for a fixed count
    span_len: int

    @property
    def units(self) -> int:
        return self.layers * self.kv_heads

    @property
    def m(self) -> int:
        return self.group * self.window


CONFIGS = {
    1: Config(1, "tiny-1layer-2kv-d64-n1k", 1, 2, 2, 64, 1024, 16, 128, 7, 1e-2,
              "f32", "normal", (4, 4), 32),
    2: Config(2, "llama3-8b-layer-n8k", 1, 8, 4, 128, 8192, 32, 512, 7, 1e-2,
              "bf16", "scaled", (16, 16), 64),
    3: Config(3, "llama3-8b-layer-n32k", 1, 8, 4, 128, 32768, 32, 2048, 7, 1e-2,
              "bf16", "scaled", (26, 26), 64),
    4: Config(4, "llama3-8b-32layer-n32k", 32, 8, 4, 128, 32768, 32, 2048, 7, 1e-2,
              "bf16", "scaled", (4, 64), 64),
    5: Config(5, "llama3-8b-4layer-n128k", 4, 8, 4, 128, 131072, 64, 4096, 7, 1e-2,
              "bf16", "student_t3", (16, 16), 64),
}


def config(cfg_id: int, **overrides) -> Config:
    """Return a named config, optionally with fields replaced (e.g. budget=1024)."""
    return dataclasses.replace(CONFIGS[cfg_id], **overrides)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = u + np.uint32(0x7FFF)
    r += lsb
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def decode(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Stored array -> exact float64 values."""
    if dtype == "bf16":
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _store(x32: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(x32) if dtype == "bf16" else np.ascontiguousarray(x32, dtype=np.float32)


def make_unit(cfg: Config, layer: int, head: int, *, n: int | None = None):
    """Draw one unit.  Returns ``(q_obs [G,w,d], K [n,d], V [n,d], spans)``.

    Arrays are float32 (f32 configs) or uint16 bfloat16 bits (bf16 configs).
    ``spans`` lists the salient ``(start, length)`` pairs, for diagnostics.
    ``n`` may override the config's token count (edge-case tests).
    """
    n = cfg.n if n is None else n
    d, G, w = cfg.head_dim, cfg.group, cfg.window
    rng = np.random.default_rng(np.random.SeedSequence([cfg.cfg_id, layer, head]))
    # 1. channel scales, 2. outlier channels
    if cfg.k_dist == "scaled":
        scales = rng.lognormal(0.0, 0.5, size=d)
        outl = rng.choice(d, size=4, replace=False)
        scales[outl] *= 8.0
    else:
        scales = None
    # 3. K, 4. V
    if cfg.k_dist == "student_t3":
        k32 = rng.standard_t(3, size=(n, d)).astype(np.float32)
    else:
        k32 = rng.standard_normal((n, d), dtype=np.float32)
        if scales is not None:
            k32 *= scales.astype(np.float32)[None, :]
    v32 = rng.standard_normal((n, d), dtype=np.float32)
    K = _store(k32, cfg.dtype)
    V = _store(v32, cfg.dtype)
    del k32, v32
    # 5. span count, 6. span slots (aligned, distinct, inside the prefix [0, n - w))
    lo, hi = cfg.span_count
    count = int(rng.integers(lo, hi + 1))
    slots_avail = max((n - w) // cfg.span_len, 1)
    count = min(count, slots_avail)
    slots = np.sort(rng.choice(slots_avail, size=count, replace=False))
    L = min(cfg.span_len, n - w) if n > w else 1
    spans = [(int(s) * cfg.span_len, L) for s in slots]
    rows = np.concatenate([np.arange(s, s + l) for s, l in spans])
    mu = decode(K[rows], cfg.dtype).mean(axis=0)
    # 7. query noise, one independent draw per (g, i)
    eps = rng.standard_normal((G, w, d))
    q64 = 0.5 * eps + 1.5 * mu[None, None, :]
    q_obs = _store(q64.astype(np.float32), cfg.dtype)
    return q_obs, K, V, spans


def make_batch(cfg: Config, units=None, *, n: int | None = None, threads: int | None = None):
    """Draw several units (default: all of them) into stacked arrays.

    ``units`` is an iterable of flat unit ids ``u = layer * kv_heads + head``.
    Returns ``(q_obs [U,G,w,d], K [U,n,d], V [U,n,d])`` in storage form.
    """
    ids = list(range(cfg.units)) if units is None else [int(u) for u in units]
    n_tok = cfg.n if n is None else n
    dt = np.uint16 if cfg.dtype == "bf16" else np.float32
    U = len(ids)
    q = np.empty((U, cfg.group, cfg.window, cfg.head_dim), dtype=dt)
    K = np.empty((U, n_tok, cfg.head_dim), dtype=dt)
    V = np.empty((U, n_tok, cfg.head_dim), dtype=dt)

    def fill(slot_uid):
        slot, uid = slot_uid
        qs, ks, vs, _ = make_unit(cfg, uid // cfg.kv_heads, uid % cfg.kv_heads, n=n)
        q[slot], K[slot], V[slot] = qs, ks, vs

    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))
    if threads <= 1 or U == 1:
        for item in enumerate(ids):
            fill(item)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, enumerate(ids)))
    return q, K, V


def make_prompt_queries(cfg: Config, q_obs: np.ndarray, K: np.ndarray, units=None, *,
                        n: int | None = None) -> np.ndarray:
    """Queries of every prompt position, for front-ends that score tokens by
    the attention of all prompt queries (accumulated attention).

    Returns ``q_all [U, G, n, d]`` in storage form whose last w positions are
    the window queries ``q_obs`` of the same units, and whose earlier positions
    follow the window's recipe (``0.5*eps + 1.5*mu`` with ``mu`` the mean of the
    unit's salient-span keys, recomputed from the same seed) with noise drawn
    from ``SeedSequence([cfg, layer, head, 1])``."""
    ids = list(range(cfg.units)) if units is None else [int(u) for u in units]
    n_tok = cfg.n if n is None else n
    U, G, w, d = q_obs.shape
    dt = np.uint16 if cfg.dtype == "bf16" else np.float32
    q_all = np.empty((U, G, n_tok, d), dtype=dt)
    for slot, uid in enumerate(ids):
        layer, head = uid // cfg.kv_heads, uid % cfg.kv_heads
        _, _, _, spans = make_unit(cfg, layer, head, n=n)
        rows = np.concatenate([np.arange(s0, s0 + l) for s0, l in spans])
        mu = decode(K[slot][rows], cfg.dtype).mean(axis=0)
        rng = np.random.default_rng(np.random.SeedSequence([cfg.cfg_id, layer, head, 1]))
        eps = rng.standard_normal((G, n_tok - w, d))
        q64 = 0.5 * eps + 1.5 * mu[None, None, :]
        q_all[slot, :, : n_tok - w] = _store(q64.astype(np.float32), cfg.dtype)
        q_all[slot, :, n_tok - w:] = q_obs[slot]
    return q_all
