"""The C-ABI library: it loads, exports every declared entry point, and
rejects bad arguments before touching the device (runs without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2411_01433_amd as P
from paper_2411_01433_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_header_matches_binding_list():
    assert declared_functions() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = B.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    syms = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    for name in declared_functions():
        assert name in syms, name
        assert getattr(L, name) is not None


def test_desc_layout_matches_header():
    # 6 int32 + 3 float + 1 uint32, no padding
    assert ctypes.sizeof(B.LayerDesc) == 40


def _desc(**kw):
    d = dict(d_model=256, d_ff=512, n_experts=8, top_k=2, group_size=32,
             max_tokens=4, t1=1.0, t2=1.0, rms_eps=1e-5, flags=0)
    d.update(kw)
    return B.LayerDesc(**d)


@pytest.mark.parametrize("bad", [
    dict(group_size=16), dict(d_model=100), dict(d_model=0), dict(d_ff=96),
    dict(n_experts=0), dict(n_experts=65), dict(top_k=0), dict(top_k=9),
    dict(top_k=9, n_experts=8), dict(max_tokens=0), dict(max_tokens=10000),
    dict(flags=1), dict(t1=float("nan")), dict(rms_eps=-1.0),
])
def test_init_rejects_bad_desc(bad):
    L = B.lib()
    desc = _desc(**bad)
    E = desc.n_experts if desc.n_experts > 0 else 1
    fake = (ctypes.c_void_p * max(E, 1))(*([0x1000] * max(E, 1)))
    out = ctypes.c_void_p(123)
    st = L.moe_layer_init(ctypes.byref(desc), ctypes.c_void_p(0x1000), fake, fake,
                          fake, None, ctypes.byref(out))
    assert st == B.MOE_EINVAL
    assert out.value is None
    assert len(L.moe_last_error()) > 0


def test_init_rejects_null_and_misaligned_pointers():
    L = B.lib()
    desc = _desc()
    fake = (ctypes.c_void_p * 8)(*([0x1000] * 8))
    out = ctypes.c_void_p()
    assert L.moe_layer_init(None, ctypes.c_void_p(0x1000), fake, fake, fake, None,
                            ctypes.byref(out)) == B.MOE_EINVAL
    assert L.moe_layer_init(ctypes.byref(desc), None, fake, fake, fake, None,
                            ctypes.byref(out)) == B.MOE_EINVAL
    nulls = (ctypes.c_void_p * 8)(*([0x1000] * 7 + [0]))
    assert L.moe_layer_init(ctypes.byref(desc), ctypes.c_void_p(0x1000), fake, nulls,
                            fake, None, ctypes.byref(out)) == B.MOE_EINVAL
    assert b"expert 7" in L.moe_last_error()
    odd = (ctypes.c_void_p * 8)(*([0x1008] * 8))
    assert L.moe_layer_init(ctypes.byref(desc), ctypes.c_void_p(0x1000), fake, fake,
                            odd, None, ctypes.byref(out)) == B.MOE_EINVAL
    assert L.moe_layer_init(ctypes.byref(desc), ctypes.c_void_p(0x1000), fake, fake,
                            fake, None, None) == B.MOE_EINVAL


def test_calls_on_invalid_handles_fail_cleanly():
    L = B.lib()
    bogus = ctypes.c_void_p(0xdead0)
    x = ctypes.c_void_p(0x1000)
    assert L.moe_set_expert_precision(bogus, 0, 1, None) == B.MOE_ESTATE
    assert L.moe_set_expert_precision(None, 0, 1, None) == B.MOE_ESTATE
    assert L.moe_decode_step(bogus, 1, x, x, None, None, None, None) == B.MOE_ESTATE
    assert L.moe_prefill(bogus, 1, x, x, None, None, None, None) == B.MOE_ESTATE
    assert L.moe_decode_step_residual(bogus, 1, x, x, x, None, None, None, None) == B.MOE_ESTATE
    assert L.moe_decode_step_prenorm(bogus, 1, x, x, None, None, None, None) == B.MOE_ESTATE
    assert L.moe_prefill_residual(bogus, 1, x, x, x, None, None, None, None) == B.MOE_ESTATE
    assert L.moe_export_packed(bogus, 0, 0, 4, x, x, None) == B.MOE_ESTATE
    assert L.moe_layer_destroy(bogus) == B.MOE_ESTATE
    assert L.moe_layer_destroy(None) == B.MOE_EINVAL
    assert L.moe_layer_share_workspace(bogus, ctypes.c_void_p(0xbeef0), None) == B.MOE_ESTATE
    assert L.moe_layer_share_workspace(bogus, bogus, None) == B.MOE_EINVAL
    assert L.moe_layer_share_workspace(None, bogus, None) == B.MOE_EINVAL
    assert b"handle" in L.moe_last_error() or b"NULL" in L.moe_last_error()


def test_quantize_rejects_bad_args():
    L = B.lib()
    p = ctypes.c_void_p(0x1000)
    assert L.moe_quantize(None, 4, 32, 4, p, p, None) == B.MOE_EINVAL
    assert L.moe_quantize(p, 4, 33, 4, p, p, None) == B.MOE_EINVAL
    assert L.moe_quantize(p, 4, 32, 3, p, p, None) == B.MOE_EINVAL
    assert L.moe_quantize(p, -1, 32, 4, p, p, None) == B.MOE_EINVAL
    assert L.moe_quantize(ctypes.c_void_p(0x1002), 4, 32, 4, p, p, None) == B.MOE_EINVAL
    assert L.moe_quantize(p, 4, 32, 4, ctypes.c_void_p(0x1008), p, None) == B.MOE_EINVAL


def test_rmsnorm_rejects_bad_args():
    L = B.lib()
    p = ctypes.c_void_p(0x1000)
    assert L.moe_rmsnorm(None, p, 4, 64, 1e-5, None) == B.MOE_EINVAL
    assert L.moe_rmsnorm(p, p, 0, 64, 1e-5, None) == B.MOE_EINVAL
    assert L.moe_rmsnorm(p, p, 4, 96, 1e-5, None) == B.MOE_EINVAL
    assert L.moe_rmsnorm(p, p, 4, 64, -1.0, None) == B.MOE_EINVAL
    assert L.moe_rmsnorm(ctypes.c_void_p(0x1004), p, 4, 64, 1e-5, None) == B.MOE_EINVAL
    assert b"aligned" in L.moe_last_error()


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        B.lib()


def test_predictor_rejects_bad_args():
    L = B.lib()
    g = (ctypes.c_void_p * 8)(*([0x1000] * 8))
    out = ctypes.c_void_p(123)
    ok = dict(d=256, E=8, K=2, p=3, T=4)

    def init(d=256, E=8, K=2, p=3, T=4, gates=g):
        return L.moe_predictor_init(d, E, K, p, T, gates, None, ctypes.byref(out))

    for bad in [dict(d=100), dict(d=0), dict(E=0), dict(E=65), dict(K=0), dict(K=9),
                dict(K=9, E=8), dict(p=0), dict(p=9), dict(T=0), dict(T=9000)]:
        kw = dict(ok)
        kw.update(bad)
        assert init(**kw) == B.MOE_EINVAL, bad
        assert out.value is None
    assert init(gates=None) == B.MOE_EINVAL
    nul = (ctypes.c_void_p * 3)(0x1000, 0, 0x1000)
    assert init(gates=nul) == B.MOE_EINVAL
    mis = (ctypes.c_void_p * 3)(0x1000, 0x1008, 0x1000)
    assert init(gates=mis) == B.MOE_EINVAL
    assert L.moe_predictor_init(256, 8, 2, 3, 4, g, None, None) == B.MOE_EINVAL


def test_predictor_invalid_handles_fail_cleanly():
    L = B.lib()
    bogus = ctypes.c_void_p(0xdead0)
    x = ctypes.c_void_p(0x1000)
    assert L.moe_predict(bogus, 1, x, x, x, None, x, x, None) == B.MOE_ESTATE
    assert L.moe_predict(None, 1, x, x, x, None, x, x, None) == B.MOE_ESTATE
    assert L.moe_predictor_destroy(bogus) == B.MOE_ESTATE
    assert L.moe_predictor_destroy(None) == B.MOE_EINVAL


def test_store_and_bind_reject_bad_args():
    L = B.lib()
    out = ctypes.c_void_p(123)
    for args in [(100, 512, 8, 4), (256, 500, 8, 4), (256, 512, 0, 4), (256, 512, 65, 4),
                 (256, 512, 8, 3), (256, 512, 8, 8)]:
        assert L.moe_store_create(*args, ctypes.byref(out)) == B.MOE_EINVAL, args
        assert out.value is None
    bogus = ctypes.c_void_p(0xdead0)
    assert L.moe_store_destroy(bogus) == B.MOE_ESTATE
    assert L.moe_store_destroy(None) == B.MOE_EINVAL
    assert L.moe_store_sizes(bogus, None, None, None) == B.MOE_ESTATE
    assert L.moe_layer_bind_expert(bogus, 0, 0, None, None, None, 0, None) == B.MOE_ESTATE
