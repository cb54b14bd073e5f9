"""Thin ctypes binding of the C ABI in include/moe.h.

Argument marshalling only: torch tensors are checked (device, dtype, shape,
contiguity, alignment) and their data pointers are passed to the library;
every step of the layer runs in the HIP kernels of libmoe.so.  There is no
fallback: if the library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")

MOE_OK, MOE_EINVAL, MOE_ENOMEM, MOE_EHIP, MOE_ESTATE, MOE_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
TAG_FP16, TAG_INT4, TAG_INT2, TAG_MISS_INT4, TAG_MISS_INT2 = 0, 1, 2, 3, 4
TAG_INT8, TAG_MISS_INT8_INT2 = 5, 6  # int8 models: int8 high copy, int2 low copy
PREC_HIGH, PREC_LOW, PREC_SKIP = 0, 1, 2

EXPORTED = (
    "moe_layer_init", "moe_set_expert_precision", "moe_decode_step",
    "moe_decode_step_residual", "moe_decode_step_prenorm", "moe_prefill",
    "moe_prefill_residual",
    "moe_export_packed", "moe_quantize", "moe_layer_enable_timing",
    "moe_layer_stage_times", "moe_layer_destroy", "moe_layer_share_workspace",
    "moe_last_error",
    "moe_predictor_init", "moe_predict", "moe_predictor_destroy",
    "moe_cache_create", "moe_cache_begin_sequence", "moe_cache_begin_token",
    "moe_cache_access", "moe_cache_contains", "moe_cache_set_mask",
    "moe_cache_clear_masks", "moe_cache_replay", "moe_cache_layer_tags",
    "moe_cache_stats", "moe_cache_destroy",
    "moe_store_create", "moe_store_sizes", "moe_store_put", "moe_store_load",
    "moe_store_destroy", "moe_layer_bind_expert", "moe_rmsnorm",
    "moe_decode_step_noalloc",
)


class MoeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"moe status {status}: {msg}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
        ("group_size", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
        ("t1", ctypes.c_float), ("t2", ctypes.c_float),
        ("rms_eps", ctypes.c_float), ("flags", ctypes.c_uint32),
    ]


class CacheDesc(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32),
        ("hi_capacity", ctypes.c_int32), ("lo_capacity", ctypes.c_int32),
        ("w_lru", ctypes.c_double), ("w_lfu", ctypes.c_double),
        ("w_lhu", ctypes.c_double), ("w_fld", ctypes.c_double),
        ("bits_hi", ctypes.c_int32), ("bits_lo", ctypes.c_int32),
        ("miss_cost", ctypes.c_double),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmoe.so (built by paper_2411_01433_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run python -m paper_2411_01433_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32p = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    L.moe_layer_init.argtypes = [ctypes.POINTER(LayerDesc), vp, ctypes.POINTER(vp),
                                 ctypes.POINTER(vp), ctypes.POINTER(vp), vp,
                                 ctypes.POINTER(vp)]
    L.moe_set_expert_precision.argtypes = [vp, i32, i32, vp]
    step = [vp, i32, vp, f32p, vp, vp, vp, vp]
    L.moe_decode_step.argtypes = step
    L.moe_decode_step_noalloc.argtypes = step
    L.moe_prefill.argtypes = step
    res = [vp, i32, vp, f32p, vp, vp, vp, vp, vp]
    L.moe_decode_step_residual.argtypes = res
    L.moe_prefill_residual.argtypes = res
    L.moe_decode_step_prenorm.argtypes = [vp, i32, f32p, vp, vp, vp, vp, vp]
    L.moe_export_packed.argtypes = [vp, i32, i32, i32, vp, vp, vp]
    L.moe_quantize.argtypes = [vp, i64, i64, i32, vp, vp, vp]
    L.moe_layer_enable_timing.argtypes = [vp, i32]
    L.moe_layer_stage_times.argtypes = [vp, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int32)]
    L.moe_layer_destroy.argtypes = [vp]
    L.moe_layer_share_workspace.argtypes = [vp, vp, vp]
    pi32 = ctypes.POINTER(ctypes.c_int32)
    L.moe_cache_create.argtypes = [ctypes.POINTER(CacheDesc), ctypes.POINTER(vp)]
    L.moe_cache_begin_sequence.argtypes = [vp]
    L.moe_cache_begin_token.argtypes = [vp]
    L.moe_cache_access.argtypes = [vp, i32, i32, i32, pi32, pi32, pi32]
    L.moe_cache_contains.argtypes = [vp, i32, i32, i32, pi32]
    L.moe_cache_set_mask.argtypes = [vp, i32, i32, i32]
    L.moe_cache_clear_masks.argtypes = [vp]
    L.moe_cache_replay.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, vp]
    L.moe_cache_layer_tags.argtypes = [vp, i32, pi32]
    L.moe_cache_stats.argtypes = [vp, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64)]
    L.moe_cache_destroy.argtypes = [vp]
    L.moe_store_create.argtypes = [i32, i32, i32, i32, ctypes.POINTER(vp)]
    L.moe_store_sizes.argtypes = [vp, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
    L.moe_store_put.argtypes = [vp, i32, vp, vp, vp, vp]
    L.moe_store_load.argtypes = [vp, i32, i32, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                 ctypes.POINTER(vp), vp]
    L.moe_store_destroy.argtypes = [vp]
    L.moe_layer_bind_expert.argtypes = [vp, i32, i32, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                        ctypes.POINTER(vp), i32, vp]
    L.moe_rmsnorm.argtypes = [vp, vp, i32, i32, ctypes.c_float, vp]
    L.moe_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name != "moe_last_error":
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int):
    if status != MOE_OK:
        raise MoeError(status, lib().moe_last_error().decode())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t, dtype, shape=None, name="tensor"):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def quantize(w, bits: int, codes, scales, stream=None):
    """Quantise an fp16 device matrix w [rows, cols] into codes / scales."""
    import torch
    rows, cols = w.shape
    _check(lib().moe_quantize(
        _ptr(w, torch.float16, None, "w"), rows, cols, bits,
        _ptr(codes, torch.uint8, (rows, cols * bits // 8), "codes"),
        _ptr(scales, torch.float16, (rows, cols // 32), "scales"), _stream(stream)))


def rmsnorm(h, x, eps: float = 1e-5, stream=None):
    """x = fp16(rmsnorm(h)) row by row (h fp32 [T, d], x fp16 [T, d])."""
    import torch
    T, d = h.shape
    _check(lib().moe_rmsnorm(_ptr(h, torch.float32, None, "h"),
                             _ptr(x, torch.float16, (T, d), "x"), T, d, eps, _stream(stream)))


class MoeLayer:
    """One MoE layer handle over borrowed fp16 device weights.

    w_router [E, d]; w1, w3: lists of E tensors [f, d]; w2: list of E [d, f].
    The tensors must outlive the layer (the library borrows them).
    """

    def __init__(self, d_model, d_ff, n_experts, top_k, max_tokens, w_router,
                 w1, w3, w2, t1=1.0, t2=1.0, rms_eps=1e-5, stream=None):
        import torch
        self.d, self.f, self.E, self.K = d_model, d_ff, n_experts, top_k
        self.max_tokens = max_tokens
        self._keep = (w_router, list(w1), list(w3), list(w2))
        desc = LayerDesc(d_model, d_ff, n_experts, top_k, 32, max_tokens,
                         t1, t2, rms_eps, 0)
        E = n_experts
        if not (len(w1) == len(w3) == len(w2) == E):
            raise ValueError("need one W1, W3 and W2 per expert")
        arr = ctypes.c_void_p * E
        p1 = arr(*[_ptr(w, torch.float16, (d_ff, d_model), "w1").value for w in w1])
        p3 = arr(*[_ptr(w, torch.float16, (d_ff, d_model), "w3").value for w in w3])
        p2 = arr(*[_ptr(w, torch.float16, (d_model, d_ff), "w2").value for w in w2])
        h = ctypes.c_void_p()
        _check(lib().moe_layer_init(ctypes.byref(desc),
                                    _ptr(w_router, torch.float16, (E, d_model), "w_router"),
                                    p1, p3, p2, _stream(stream), ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    def set_expert_precision(self, expert: int, tag: int, stream=None):
        _check(lib().moe_set_expert_precision(self._h, expert, tag, _stream(stream)))

    def _outs(self, T, topk_idx, topk_w, prec_used):
        import torch
        return (_ptr(topk_idx, torch.int32, (T, self.K), "topk_idx"),
                _ptr(topk_w, torch.float32, (T, self.K), "topk_w"),
                _ptr(prec_used, torch.int8, (T, self.K), "prec_used"))

    def _step(self, fn, x, y, topk_idx, topk_w, prec_used, stream):
        import torch
        T = x.shape[0]
        _check(fn(self._h, T, _ptr(x, torch.float16, (T, self.d), "x"),
                  _ptr(y, torch.float32, (T, self.d), "y"),
                  *self._outs(T, topk_idx, topk_w, prec_used), _stream(stream)))

    def _step_res(self, fn, x, h, x_next, topk_idx, topk_w, prec_used, stream):
        import torch
        T = x.shape[0]
        _check(fn(self._h, T, _ptr(x, torch.float16, (T, self.d), "x"),
                  _ptr(h, torch.float32, (T, self.d), "h"),
                  _ptr(x_next, torch.float16, (T, self.d), "x_next"),
                  *self._outs(T, topk_idx, topk_w, prec_used), _stream(stream)))

    def decode_step(self, x, y, topk_idx=None, topk_w=None, prec_used=None, stream=None):
        self._step(lib().moe_decode_step, x, y, topk_idx, topk_w, prec_used, stream)

    def decode_step_noalloc(self, x, y, topk_idx=None, topk_w=None, prec_used=None,
                            stream=None):
        """moe_decode_step_noalloc: the decode step with the static scratch."""
        self._step(lib().moe_decode_step_noalloc, x, y, topk_idx, topk_w, prec_used, stream)

    def prefill(self, x, y, topk_idx=None, topk_w=None, prec_used=None, stream=None):
        self._step(lib().moe_prefill, x, y, topk_idx, topk_w, prec_used, stream)

    def decode_step_residual(self, x, h, x_next, topk_idx=None, topk_w=None,
                             prec_used=None, stream=None):
        self._step_res(lib().moe_decode_step_residual, x, h, x_next, topk_idx,
                       topk_w, prec_used, stream)

    def decode_step_prenorm(self, h, x, topk_idx=None, topk_w=None, prec_used=None,
                            stream=None):
        """moe_decode_step_prenorm: x = fp16(rmsnorm(h)) formed by the step, then
        h += MoE(x) (h is the residual stream, x an output)."""
        import torch
        T = h.shape[0]
        _check(lib().moe_decode_step_prenorm(
            self._h, T, _ptr(h, torch.float32, (T, self.d), "h"),
            _ptr(x, torch.float16, (T, self.d), "x"),
            *self._outs(T, topk_idx, topk_w, prec_used), _stream(stream)))

    def prefill_residual(self, x, h, x_next, topk_idx=None, topk_w=None,
                         prec_used=None, stream=None):
        self._step_res(lib().moe_prefill_residual, x, h, x_next, topk_idx,
                       topk_w, prec_used, stream)

    def export_packed(self, expert: int, matrix: int, bits: int, codes, scales,
                      stream=None):
        import torch
        rows, cols = (self.f, self.d) if matrix < 2 else (self.d, self.f)
        _check(lib().moe_export_packed(
            self._h, expert, matrix, bits,
            _ptr(codes, torch.uint8, (rows, cols * bits // 8), "codes"),
            _ptr(scales, torch.float16, (rows, cols // 32), "scales"), _stream(stream)))

    def bind_expert(self, expert: int, tag: int, w=None, q=None, s=None, low_bits=0,
                    stream=None):
        """Point an expert at caller-owned device copies: w = [W1, W3, W2] fp16,
        q / s = codes / scales of the low copy (uint8 / fp16, layout as quantize)."""
        import torch

        def arr(ts, dtype, name):
            if ts is None:
                return None
            shapes = [(self.f, self.d), (self.f, self.d), (self.d, self.f)]
            ptrs = []
            for m, t in enumerate(ts):
                rows, cols = shapes[m]
                shp = {torch.float16: (rows, cols)}.get(dtype)
                if name == "q":
                    shp = (rows, cols * low_bits // 8)
                elif name == "s":
                    shp = (rows, cols // 32)
                ptrs.append(_ptr(t, dtype, shp, f"{name}[{m}]").value)
            return (ctypes.c_void_p * 3)(*ptrs)
        _check(lib().moe_layer_bind_expert(self._h, expert, tag, arr(w, torch.float16, "w"),
                                           arr(q, torch.uint8, "q"), arr(s, torch.float16, "s"),
                                           low_bits, _stream(stream)))

    def enable_timing(self, on: bool = True):
        _check(lib().moe_layer_enable_timing(self._h, 1 if on else 0))

    def stage_times(self):
        """(summed ms per stage [route, up, down, combine], n_calls); resets."""
        ms = (ctypes.c_double * 4)()
        n = ctypes.c_int32()
        _check(lib().moe_layer_stage_times(self._h, ms, ctypes.byref(n)))
        return list(ms), n.value

    def share_workspace(self, owner: "MoeLayer", stream=None):
        """Run this layer on owner's per-call workspace and free its own (the
        layers of a stack run one after another).  Equal d, f, top_k and
        max_tokens; owner is kept alive by this layer."""
        _check(lib().moe_layer_share_workspace(self._h, owner._h, _stream(stream)))
        self._ws_owner = owner

    def destroy(self):
        if self._h is not None and self._h.value:
            _check(lib().moe_layer_destroy(self._h))
        self._h = None
        self._keep = None
        self._ws_owner = None

    def __del__(self):
        try:
            if getattr(self, "_h", None) is not None and self._h.value:
                lib().moe_layer_destroy(self._h)
        except Exception:
            pass


class MoePredictor:
    """Stacking Computer handle: the gates of the next p layers (a list of p
    fp16 device tensors [E, d], copied into one stacked array at creation)."""

    def __init__(self, d_model, n_experts, top_k, max_tokens, w_router_next, stream=None):
        import torch
        self.d, self.E, self.K, self.p = d_model, n_experts, top_k, len(w_router_next)
        self.max_tokens = max_tokens
        arr = ctypes.c_void_p * self.p
        gates = arr(*[_ptr(w, torch.float16, (n_experts, d_model), "w_router_next").value
                      for w in w_router_next])
        h = ctypes.c_void_p()
        _check(lib().moe_predictor_init(d_model, n_experts, top_k, self.p, max_tokens,
                                        gates, _stream(stream), ctypes.byref(h)))
        self._h = h

    def predict(self, x, cached, pred_idx, first_miss, preload, pred_w=None, stream=None):
        """x [T, d] fp16; cached int64 [p] (bit masks); pred_idx int32 [T, p, K];
        first_miss int32 [1]; preload int64 [1]; pred_w fp32 [T, p, K] or None."""
        import torch
        T = x.shape[0]
        _check(lib().moe_predict(
            self._h, T, _ptr(x, torch.float16, (T, self.d), "x"),
            _ptr(cached, torch.int64, (self.p,), "cached"),
            _ptr(pred_idx, torch.int32, (T, self.p, self.K), "pred_idx"),
            _ptr(pred_w, torch.float32, (T, self.p, self.K), "pred_w"),
            _ptr(first_miss, torch.int32, (1,), "first_miss"),
            _ptr(preload, torch.int64, (1,), "preload"), _stream(stream)))

    def destroy(self):
        if self._h is not None and self._h.value:
            _check(lib().moe_predictor_destroy(self._h))
        self._h = None

    def __del__(self):
        try:
            if getattr(self, "_h", None) is not None and self._h.value:
                lib().moe_predictor_destroy(self._h)
        except Exception:
            pass


class MoeCache:
    """Mixed-precision expert cache manager (host side, no device work)."""

    def __init__(self, n_layers, n_experts, hi_capacity, lo_capacity, w_lru, w_lfu, w_lhu,
                 w_fld, bits_hi=16, bits_lo=4, miss_cost=1.0):
        self.n_layers, self.n_experts = n_layers, n_experts
        desc = CacheDesc(n_layers, n_experts, hi_capacity, lo_capacity, w_lru, w_lfu, w_lhu,
                         w_fld, bits_hi, bits_lo, miss_cost)
        h = ctypes.c_void_p()
        _check(lib().moe_cache_create(ctypes.byref(desc), ctypes.byref(h)))
        self._h = h

    def begin_sequence(self):
        _check(lib().moe_cache_begin_sequence(self._h))

    def begin_token(self):
        _check(lib().moe_cache_begin_token(self._h))

    def access(self, layer, expert, high):
        """(hit, evicted (layer, expert) or None)."""
        hit, el, ee = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().moe_cache_access(self._h, layer, expert, 1 if high else 0,
                                      ctypes.byref(hit), ctypes.byref(el), ctypes.byref(ee)))
        return bool(hit.value), (None if el.value < 0 else (el.value, ee.value))

    def contains(self, layer, expert, high):
        v = ctypes.c_int32()
        _check(lib().moe_cache_contains(self._h, layer, expert, 1 if high else 0,
                                        ctypes.byref(v)))
        return bool(v.value)

    def set_mask(self, layer, expert, masked):
        _check(lib().moe_cache_set_mask(self._h, layer, expert, 1 if masked else 0))

    def clear_masks(self):
        _check(lib().moe_cache_clear_masks(self._h))

    def replay(self, tokens, layers, experts, highs, new_sequence=None):
        """Replay a trace (numpy arrays); returns (hits int32 [n], evicted int32 [n],
        key layer * n_experts + expert or -1)."""
        import numpy as np
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        n = t.shape[0]
        arrs = [np.ascontiguousarray(a, dtype=np.int32) for a in (layers, experts, highs)]
        if any(a.shape != (n,) for a in arrs):
            raise ValueError("trace arrays must have the same length")
        ns = None if new_sequence is None else np.ascontiguousarray(new_sequence, dtype=np.uint8)
        if ns is not None and ns.shape != (n,):
            raise ValueError("new_sequence must have the trace's length")
        hits = np.empty(n, np.int32)
        ev = np.empty(n, np.int32)
        p = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
        _check(lib().moe_cache_replay(self._h, n, p(t), p(arrs[0]), p(arrs[1]), p(arrs[2]),
                                      p(ns), p(hits), p(ev)))
        return hits, ev

    def layer_tags(self, layer):
        import numpy as np
        tags = np.empty(self.n_experts, np.int32)
        _check(lib().moe_cache_layer_tags(self._h, layer,
                                          tags.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return tags

    def stats(self):
        """(penalty, hi_misses, lo_misses, hits)."""
        pen = ctypes.c_double()
        a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().moe_cache_stats(self._h, ctypes.byref(pen), ctypes.byref(a),
                                     ctypes.byref(b), ctypes.byref(c)))
        return pen.value, a.value, b.value, c.value

    def destroy(self):
        if self._h is not None and self._h.value:
            _check(lib().moe_cache_destroy(self._h))
        self._h = None

    def __del__(self):
        try:
            if getattr(self, "_h", None) is not None and self._h.value:
                lib().moe_cache_destroy(self._h)
        except Exception:
            pass


class MoeStore:
    """Pinned host storage of one layer's experts (fp16 + one low copy)."""

    def __init__(self, d_model, d_ff, n_experts, low_bits):
        self.d, self.f, self.E, self.bits = d_model, d_ff, n_experts, low_bits
        h = ctypes.c_void_p()
        _check(lib().moe_store_create(d_model, d_ff, n_experts, low_bits, ctypes.byref(h)))
        self._h = h
        a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().moe_store_sizes(h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
        self.fp16_bytes, self.code_bytes, self.scale_bytes = a.value, b.value, c.value

    def put(self, expert, w1, w3, w2, stream=None):
        import torch
        _check(lib().moe_store_put(
            self._h, expert, _ptr(w1, torch.float16, (self.f, self.d), "w1"),
            _ptr(w3, torch.float16, (self.f, self.d), "w3"),
            _ptr(w2, torch.float16, (self.d, self.f), "w2"), _stream(stream)))

    def slots(self, high, device="cuda"):
        """Device buffers for one expert copy: ([W1, W3, W2] fp16) or
        ([codes x3], [scales x3])."""
        import torch
        d, f, b = self.d, self.f, self.bits
        shapes = [(f, d), (f, d), (d, f)]
        if high:
            return [torch.empty(s_, dtype=torch.float16, device=device) for s_ in shapes]
        return ([torch.empty((r, c * b // 8), dtype=torch.uint8, device=device) for r, c in shapes],
                [torch.empty((r, c // 32), dtype=torch.float16, device=device) for r, c in shapes])

    def load(self, expert, high, dst, stream=None):
        """dst: [W1, W3, W2] (high) or (codes[3], scales[3]) from slots()."""
        V3 = ctypes.c_void_p * 3
        if high:
            w = V3(*[t.data_ptr() for t in dst])
            q = s_ = None
        else:
            w = None
            q = V3(*[t.data_ptr() for t in dst[0]])
            s_ = V3(*[t.data_ptr() for t in dst[1]])
        _check(lib().moe_store_load(self._h, expert, 1 if high else 0, w, q, s_,
                                    _stream(stream)))

    def destroy(self):
        if self._h is not None and self._h.value:
            _check(lib().moe_store_destroy(self._h))
        self._h = None

    def __del__(self):
        try:
            if getattr(self, "_h", None) is not None and self._h.value:
                lib().moe_store_destroy(self._h)
        except Exception:
            pass
