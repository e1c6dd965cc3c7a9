"""The C ABI library on the CPU: it loads, exports every declared symbol, and
rejects bad arguments on the host before launching anything."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import paper_2605_31105_amd as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "grkv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(grkv_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(G.lib_path()):
        pytest.skip("libgrkv.so not built")
    return G.lib()


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert set(names) == set(G.EXPORTED_SYMBOLS)
    for name in names:
        assert hasattr(L, name), name


def test_defaults_and_status_strings(L):
    o = G.Options()
    L.grkv_default_options(ctypes.byref(o))
    assert (o.n_sink, o.fix_window, o.causal_window) == (4, 1, 1)
    assert abs(o.beta - 0.1) < 1e-7
    for st in (0, -1, -2, -3, -4, 7):
        assert len(G.status_string(st)) > 0


def _call(L, U=2, Gq=4, d=128, dt=0, n=8192, w=32, c=512, k=7, lam=1e-2, opt=None,
          ws_bytes=None, ws_ptr=4096, nullq=False):
    prob = G.Problem(U, Gq, d, dt)
    fake = ctypes.c_void_p(4096)   # never dereferenced: validation fails first
    need = L.grkv_workspace_bytes(ctypes.byref(prob), n, w, c)
    outs = G.Outputs(4096, 4096, 4096, 0, ws_ptr,
                     (need if ws_bytes is None else ws_bytes))
    return L.grkv_compress(None if nullq else fake, fake, fake, n, w, c, k, lam, None,
                           ctypes.byref(prob), ctypes.byref(opt) if opt else None,
                           ctypes.byref(outs))


@pytest.mark.parametrize("kw,code", [
    (dict(nullq=True), G.GRKV_ERR_INVALID),
    (dict(U=0), G.GRKV_ERR_INVALID),
    (dict(Gq=0), G.GRKV_ERR_INVALID),
    (dict(dt=7), G.GRKV_ERR_INVALID),
    (dict(w=0), G.GRKV_ERR_INVALID),
    (dict(c=16), G.GRKV_ERR_INVALID),
    (dict(c=9000), G.GRKV_ERR_INVALID),
    (dict(k=4), G.GRKV_ERR_INVALID),
    (dict(k=0), G.GRKV_ERR_INVALID),
    (dict(lam=-1.0), G.GRKV_ERR_INVALID),
    (dict(lam=math.nan), G.GRKV_ERR_INVALID),
    (dict(lam=math.inf), G.GRKV_ERR_INVALID),
    (dict(opt=G.Options(4, 1.5, 1, 1)), G.GRKV_ERR_INVALID),
    (dict(opt=G.Options(-1, 0.1, 1, 1)), G.GRKV_ERR_INVALID),
    (dict(d=96), G.GRKV_ERR_UNSUPPORTED),
    (dict(Gq=8, w=64), G.GRKV_ERR_UNSUPPORTED),
    (dict(ws_bytes=1024), G.GRKV_ERR_WORKSPACE),
    (dict(ws_ptr=4096 + 8), G.GRKV_ERR_INVALID),
])
def test_invalid_arguments_rejected_before_launch(L, kw, code):
    assert _call(L, **kw) == code


def test_workspace_size_and_layout(L):
    def wb(**kw):
        a = dict(U=8, Gq=4, d=128, dt=0, n=8192, w=32, c=512)
        a.update(kw)
        return G.workspace_bytes(a["U"], a["Gq"], a["d"], a["dt"], a["n"], a["w"], a["c"])
    base = wb()
    assert base > 0
    assert wb(n=32768) > base and wb(c=1024) > base and wb(U=16) > base
    assert wb(d=96) == 0 and wb(c=4) == 0
    lay = G.workspace_layout(8, 4, 128, 0, 8192, 32, 512)
    offs = [lay.lse, lay.y, lay.score, lay.pooled, lay.fixed, lay.resid, lay.gram, lay.z]
    assert len(set(offs)) == len(offs)
    assert all(o % 256 == 0 and o < lay.total for o in offs)
    assert lay.total == base


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    q = torch.zeros(1, 1, 4, 64)
    K = torch.zeros(1, 16, 64)
    with pytest.raises(ValueError):
        G.compress(q, K, K, 4, 8, 7, 1e-2)


def _call_kv(L, U=2, Gq=4, d=128, dt=0, n=8192, w=32, c=512, k=7, lam=1e-2, kopt=None,
             ws_bytes=None, null_kstar=False, steps_ws=1):
    prob = G.Problem(U, Gq, d, dt)
    fake = ctypes.c_void_p(4096)   # never dereferenced: validation fails first
    need = L.grkv_workspace_bytes_kv(ctypes.byref(prob), n, w, c, steps_ws)
    outs = G.Outputs(4096, 4096, 4096, 0, 4096, (need if ws_bytes is None else ws_bytes))
    return L.grkv_compress_kv(fake, fake, fake, n, w, c, k, lam, None, ctypes.byref(prob), None,
                              ctypes.byref(outs), ctypes.byref(kopt) if kopt else None,
                              None if null_kstar else fake, None)


@pytest.mark.parametrize("kw,code", [
    (dict(null_kstar=True), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(-1.0, 10, 1e-5, 1)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(math.nan, 10, 1e-5, 1)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, -1, 1e-5, 1)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, 5000, 1e-5, 1)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, 10, -1.0, 1)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, 10, 1e-5, 0)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, 10, 1e-5, 17)), G.GRKV_ERR_INVALID),
    (dict(kopt=G.KeyOptions(1e-2, 10, 1e-5, 2), ws_bytes=None, steps_ws=1), G.GRKV_ERR_WORKSPACE),
    (dict(c=16), G.GRKV_ERR_INVALID),
    (dict(dt=1), G.GRKV_ERR_UNSUPPORTED),
    (dict(Gq=8, w=32), G.GRKV_ERR_UNSUPPORTED),
    (dict(ws_bytes=1024), G.GRKV_ERR_WORKSPACE),
])
def test_key_step_invalid_arguments_rejected_before_launch(L, kw, code):
    assert _call_kv(L, **kw) == code


def test_key_step_workspace_and_defaults(L):
    base = G.workspace_bytes(8, 4, 128, 0, 8192, 32, 512)
    kv = G.workspace_bytes_kv(8, 4, 128, 0, 8192, 32, 512)
    assert G.workspace_bytes_kv(8, 4, 128, 0, 8192, 32, 512, steps=2) > kv
    assert G.workspace_bytes_kv(8, 4, 128, 0, 8192, 32, 512, steps=0) == 0
    assert kv > base
    assert G.workspace_bytes_kv(8, 4, 128, 1, 8192, 32, 512) == 0     # fp32: no key step
    assert G.workspace_bytes_kv(8, 8, 128, 0, 8192, 32, 512) == 0     # m = 256
    ko = G.KeyOptions()
    L.grkv_default_key_options(ctypes.byref(ko), ctypes.c_float(0.25))
    assert (ko.lambda_k, ko.max_iter, ko.steps) == (0.25, 64, 1) and abs(ko.tol - 1e-5) < 1e-12


@pytest.mark.parametrize("kw,code", [
    (dict(nullk=True), G.GRKV_ERR_INVALID),
    (dict(c=0), G.GRKV_ERR_INVALID),
    (dict(c=9000, n=8192), G.GRKV_ERR_INVALID),
    (dict(dt=1), G.GRKV_ERR_UNSUPPORTED),
    (dict(d=96), G.GRKV_ERR_UNSUPPORTED),
    (dict(c=8193, n=20000), G.GRKV_ERR_UNSUPPORTED),
    (dict(U=0), G.GRKV_ERR_INVALID),
])
def test_carrier_stats_invalid_arguments_rejected_before_launch(L, kw, code):
    a = dict(U=2, Gq=4, d=128, dt=0, n=8192, c=512, nullk=False)
    a.update(kw)
    prob = G.Problem(a["U"], a["Gq"], a["d"], a["dt"])
    fake = ctypes.c_void_p(4096)   # never dereferenced: validation fails first
    st = L.grkv_carrier_stats(None if a["nullk"] else fake, a["n"], a["c"], ctypes.byref(prob),
                              fake, None, None, fake, None, fake, None)
    assert st == code


@pytest.mark.parametrize("args", [(32, 8, 2048, 32, 32768, 0.5), (4, 2, 256, 32, 2048, 0.5),
                                  (4, 1, 40, 32, 100, 0.1), (1, 4, 500, 16, 1000, 0.5),
                                  (7, 3, 300, 8, 5000, 0.3)])
def test_pyramid_budgets_match_the_oracle(L, args):
    # a host function: no GPU needed
    from oracle import grkv_frontend_oracle as FO
    got = G.pyramid_budgets(*args)
    want = FO.pyramid_budgets(*args[:5], ratio=args[5])
    assert np.array_equal(got, want)


def test_front_end_arguments_rejected(L):
    out = (ctypes.c_int32 * 8)()
    assert L.grkv_pyramid_budgets(0, 8, 100, 8, 1000, ctypes.c_float(0.5), out) == G.GRKV_ERR_INVALID
    assert L.grkv_pyramid_budgets(2, 4, 4, 8, 1000, ctypes.c_float(0.5), out) == G.GRKV_ERR_INVALID
    assert L.grkv_pyramid_budgets(2, 4, 100, 8, 1000, ctypes.c_float(1.5), out) == G.GRKV_ERR_INVALID
    fake = ctypes.c_void_p(4096)
    assert L.grkv_adaptive_budgets(fake, 1, 8, 1000, 8, 4, None, fake) == G.GRKV_ERR_INVALID
    assert L.grkv_adaptive_budgets(fake, 1, 200, 1000, 8, 100, None, fake) == G.GRKV_ERR_UNSUPPORTED
    prob = G.Problem(2, 4, 128, 0)
    b = (ctypes.c_int32 * 2)(64, 16)   # second budget below the window
    assert L.grkv_workspace_bytes_ragged(ctypes.byref(prob), 2048, 32, b) == 0
    b = (ctypes.c_int32 * 2)(64, 128)
    assert L.grkv_workspace_bytes_ragged(ctypes.byref(prob), 2048, 32, b) > 0


def _call_noalloc(L, U=2, Gq=4, d=128, dt=0, n=8192, w=32, c=512, k=7, lam=1e-2, opt=None,
                  nullq=False):
    prob = G.Problem(U, Gq, d, dt)
    fake = ctypes.c_void_p(4096)   # never dereferenced: validation fails first
    outs = G.Outputs(4096, 4096, 4096, 0, None, 0)
    return L.grkv_compress_noalloc(None if nullq else fake, fake, fake, n, w, c, k, lam, None,
                                   ctypes.byref(prob), ctypes.byref(opt) if opt else None,
                                   ctypes.byref(outs))


@pytest.mark.parametrize("kw,code", [
    (dict(nullq=True), G.GRKV_ERR_INVALID),
    (dict(U=0), G.GRKV_ERR_INVALID),
    (dict(c=16), G.GRKV_ERR_INVALID),
    (dict(k=4), G.GRKV_ERR_INVALID),
    (dict(lam=math.nan), G.GRKV_ERR_INVALID),
    (dict(opt=G.Options(4, 1.5, 1, 1)), G.GRKV_ERR_INVALID),
    (dict(d=96), G.GRKV_ERR_UNSUPPORTED),
    # 256 units of the 32k Llama-shaped workload need ~243 MiB > the 64 MiB array
    (dict(U=256, n=32768, c=2048), G.GRKV_ERR_WORKSPACE),
    (dict(U=8, n=131072, w=64, c=4096), G.GRKV_ERR_WORKSPACE),
])
def test_noalloc_rejects_before_touching_the_device(L, kw, code):
    assert _call_noalloc(L, **kw) == code


def test_noalloc_scratch_holds_a_one_layer_32k_call(L):
    prob = G.Problem(8, 4, 128, G.GRKV_BF16)
    need = L.grkv_workspace_bytes(ctypes.byref(prob), 32768, 32, 2048)
    assert 0 < need <= G.NOALLOC_SCRATCH_BYTES
