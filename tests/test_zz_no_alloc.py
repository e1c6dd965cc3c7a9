"""The allocation-free entry point (grkv_compress_noalloc) against
grkv_compress, through the C ABI: two calls in a row on the library's scratch
array, the second with a smaller input, each matching the workspace entry
point's outputs bit for bit (same kernels, same launch sequence).  The
refusal of shapes beyond the scratch array is a host check, tested on the CPU
with the other argument errors."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _dev(arr):
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()


def _outputs(U, c, d):
    import paper_2605_31105_amd as G
    return G.Result(idx=torch.empty((U, c), dtype=torch.int32, device="cuda"),
                    k_out=torch.empty((U, c, d), dtype=torch.bfloat16, device="cuda"),
                    v_out=torch.empty((U, c, d), dtype=torch.float32, device="cuda"),
                    stats=torch.empty((U, 4), dtype=torch.float32, device="cuda"),
                    workspace=None, shape=())


def _same(a, b):
    for k in ("idx", "k_out", "v_out", "stats"):
        x, y = getattr(a, k), getattr(b, k)
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), k


def test_noalloc_matches_workspace_entry_point_twice():
    import paper_2605_31105_amd as G
    # first call: one 8k layer (8 units); second: 2 units of a 2k cache
    for cfg in (W.config(2), W.config(2, layers=1, kv_heads=2, n=2048, budget=256)):
        print("case noalloc", cfg.units, cfg.n, cfg.budget, flush=True)
        assert G.workspace_bytes(cfg.units, cfg.group, cfg.head_dim, G.GRKV_BF16, cfg.n,
                                 cfg.window, cfg.budget) <= G.NOALLOC_SCRATCH_BYTES
        q, K, V = (_dev(a) for a in W.make_batch(cfg))
        ref = G.compress(q, K, V, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam)
        got = G.compress_noalloc(q, K, V, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam,
                                 out=_outputs(cfg.units, cfg.budget, cfg.head_dim))
        torch.cuda.synchronize()
        _same(ref, got)
        assert torch.all(got.stats[:, 3] == 0)
