"""The seeded input generator: determinism, bfloat16 rounding, span recipe."""
import numpy as np

import workloads as W


def test_bf16_round_nearest_even():
    f = np.array([1.0, 1.00390625, 1.005859375, 1.0078125 + 2 ** -8, -2.5, 3.0e38, 1e-40],
                 dtype=np.float32)
    b = W.f32_to_bf16_bits(f)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> ties to even (1.0)
    assert b[0] == 0x3F80 and b[1] == 0x3F80
    # 1 + 2^-8 + 2^-9 rounds up to 1 + 2^-7
    assert b[2] == 0x3F81
    # 1 + 2^-7 + 2^-8 is halfway between 1+2^-7 (odd) and 1+2^-6 -> even
    assert b[3] == 0x3F82
    assert b[4] == 0xC020
    np.testing.assert_array_equal(W.bf16_bits_to_f32(b[:2]), [1.0, 1.0])
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    y = W.bf16_bits_to_f32(W.f32_to_bf16_bits(x))
    assert np.all(np.abs(y - x) <= np.abs(x) * 2.0 ** -8)


def test_determinism_and_unit_independence():
    cfg = W.config(2, n=512, budget=128)
    a = W.make_batch(cfg, units=[3, 5])
    b = W.make_batch(cfg, units=[5])
    np.testing.assert_array_equal(a[1][1], b[1][0])
    np.testing.assert_array_equal(a[2][1], b[2][0])
    np.testing.assert_array_equal(a[0][1], b[0][0])
    c = W.make_batch(cfg, units=[3, 5], threads=1)
    for x, y in zip(a, c):
        np.testing.assert_array_equal(x, y)


def test_shapes_and_spans():
    for cid in (1, 2, 3, 4, 5):
        cfg = W.CONFIGS[cid]
        assert cfg.m == cfg.group * cfg.window
    cfg = W.config(3)
    q, K, V, spans = W.make_unit(cfg, 0, 1)
    assert q.shape == (4, 32, 128) and K.shape == (32768, 128) and q.dtype == np.uint16
    cover = sum(l for _, l in spans)
    assert cover == 26 * 64 and abs(cover / cfg.n - 0.05) < 0.002
    assert all(s % 64 == 0 and s + l <= cfg.n - cfg.window for s, l in spans)
    cfg4 = W.config(4)
    counts = {len(W.make_unit(W.config(4, n=4096), L, 0)[3]) for L in range(12)}
    assert min(counts) >= 4 and max(counts) <= 64 and len(counts) > 3
