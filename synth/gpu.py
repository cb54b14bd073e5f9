"""Device-side generation of the keyed fp16 tensors (same values as
synth.gen.normal_fp16, generated in HBM).  Input generation only."""
from __future__ import annotations

import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "synth_gpu.hip")
LIB = os.path.join(HERE, "libsynth.so")

_lib = None
_tables = {}


def build() -> str:
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-x", "hip", SRC, "-o", LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {SRC}:\n{r.stderr}")
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise ImportError(f"{LIB} missing: build it with synth.gpu.build()")
        L = ctypes.CDLL(LIB)
        L.synth_normal_fp16.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.synth_normal_fp16.restype = ctypes.c_int
        _lib = L
    return _lib


def _table(std: float, device):
    import torch
    from .gen import normal_table
    k = (float(std), str(device))
    if k not in _tables:
        t = torch.from_numpy(normal_table(std).view("uint16").astype("int16"))
        _tables[k] = t.to(device)
    return _tables[k]


def normal_fp16_(out, key: int, std: float, start: int = 0, stream=None):
    """Fill the contiguous fp16 device tensor ``out`` with stream elements
    [start, start + out.numel()) of the keyed generator."""
    import torch
    assert out.dtype == torch.float16 and out.is_contiguous() and out.is_cuda
    tab = _table(std, out.device)
    s = torch.cuda.current_stream() if stream is None else stream
    rc = _load().synth_normal_fp16(ctypes.c_uint64(key), ctypes.c_void_p(tab.data_ptr()),
                                   ctypes.c_void_p(out.data_ptr()), out.numel(), start,
                                   ctypes.c_void_p(s.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"synth_normal_fp16 failed ({rc})")
    return out
