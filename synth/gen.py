"""Counter-based generator of fp16 N(0, std) tensors, keyed per tensor.

Definition (identical in numpy here and in the HIP kernel in synth_gpu.hip):

* ``mix64`` is the SplitMix64 output function (Steele, Lea and Flood,
  "Fast splittable pseudorandom number generators", OOPSLA 2014):
  z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
  z *= 0x94D049BB133111EB; z ^= z >> 31   (all mod 2**64).
* A tensor is named by the key (seed, layer, tensor_id, expert).  Its 64-bit
  stream key is  k = mix64(mix64(mix64(mix64(SEED_MIX ^ seed) ^ layer)
  ^ tensor_id) ^ expert).
* Word c of the stream is  r_c = mix64(k + (c + 1) * GOLDEN)  (SplitMix64's
  c-th output from state k).  Element i of the tensor is the 16-bit lane
  j = i % 4 of word c = i // 4:  u_i = (r_c >> 16 j) & 0xFFFF.
* The value is  table[u_i]  where  table[u] = fp16(std * Phi^-1((u + 0.5)
  / 65536)), computed once in float64 and rounded to fp16 (RNE).

So every value is an equiprobable quantile of N(0, std), already fp16, and
both sides only index the same table: there is no transcendental function
evaluated on the device and nothing that could round differently.
"""
from __future__ import annotations

import functools

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
MIX_C1 = np.uint64(0xBF58476D1CE4E5B9)
MIX_C2 = np.uint64(0x94D049BB133111EB)
SEED_MIX = 0x2411_0143_3B0B_B17  # arbitrary fixed salt for the key chain

# tensor ids of the key (seed, layer, tensor_id, expert)
TENSOR_X = 1
TENSOR_WG = 2
TENSOR_W1 = 3
TENSOR_W3 = 4
TENSOR_W2 = 5
TENSOR_XMEAN = 6
TENSOR_TAGS = 7

_M64 = (1 << 64) - 1


def _mix64_int(z: int) -> int:
    z &= _M64
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & _M64
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & _M64
    z ^= z >> 31
    return z


def tensor_key(seed: int, layer: int, tensor_id: int, expert: int) -> int:
    """64-bit stream key of one named tensor (see module docstring)."""
    k = _mix64_int(SEED_MIX ^ (seed & _M64))
    k = _mix64_int(k ^ (layer & _M64))
    k = _mix64_int(k ^ (tensor_id & _M64))
    k = _mix64_int(k ^ (expert & _M64))
    return k


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * MIX_C1
    z = z ^ (z >> np.uint64(27))
    z = z * MIX_C2
    z = z ^ (z >> np.uint64(31))
    return z


def uniform_u16(key: int, n: int, start: int = 0) -> np.ndarray:
    """u_i for i in [start, start + n) of the stream named by ``key``."""
    if n <= 0:
        return np.zeros(0, dtype=np.uint16)
    c0 = start // 4
    c1 = (start + n + 3) // 4
    with np.errstate(over="ignore"):
        c = np.arange(c0, c1, dtype=np.uint64)
        z = np.uint64(key) + (c + np.uint64(1)) * GOLDEN
        r = _mix64_np(z)
    u = r.astype("<u8").view("<u2")
    off = start - 4 * c0
    return u[off:off + n].copy()


@functools.lru_cache(maxsize=None)
def normal_table(std: float) -> np.ndarray:
    """The 65536-entry fp16 quantile table of N(0, std)."""
    from scipy.special import ndtri

    p = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
    t = (ndtri(p) * float(std)).astype(np.float16)
    t.setflags(write=False)
    return t


def normal_fp16(seed: int, layer: int, tensor_id: int, expert: int,
                shape, std: float, start: int = 0) -> np.ndarray:
    """fp16 tensor of the given shape, N(0, std) quantiles, keyed as above.

    ``start`` offsets into the flat stream, so a row block of a large tensor
    can be generated alone: rows [r0, r1) of an [R, C] tensor are
    ``normal_fp16(..., shape=(r1 - r0, C), start=r0 * C)``.
    """
    n = int(np.prod(shape)) if len(shape) else 1
    u = uniform_u16(tensor_key(seed, layer, tensor_id, expert), n, start)
    return normal_table(std)[u].reshape(shape)
