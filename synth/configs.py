"""The synthetic workloads: shapes, seeds, tags and input recipes.

Shapes come from the paper's model table (Mixtral-8x7B: d_model 4096,
d_ff 14336, 8 experts, top-2; Phi-MoE: d_model 4096, d_ff 6400, 16 experts,
top-2; both 32 layers).  Values are synthetic (no trained weights exist
here): hidden states N(0, 1) and weights N(0, 0.02), fp16, drawn from the
keyed generator in ``synth.gen``.  Nothing here computes any part of the
MoE method; precision maps are seeded permutations of expert ids.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .gen import (TENSOR_TAGS, TENSOR_W1, TENSOR_W2, TENSOR_W3, TENSOR_WG,
                  TENSOR_X, TENSOR_XMEAN, normal_fp16, tensor_key,
                  uniform_u16)

# tag values (mirrors the library's enum; plain data, no method arithmetic)
TAG_FP16, TAG_INT4, TAG_INT2, TAG_MISS_INT4, TAG_MISS_INT2 = 0, 1, 2, 3, 4
TAG_INT8, TAG_MISS_INT8_INT2 = 5, 6

W_STD = 0.02
X_STD = 1.0


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    d_model: int
    d_ff: int
    n_experts: int
    top_k: int
    n_tokens: int
    n_layers: int = 1
    t1: float = 1.0          # Eq. 2 thresholds
    t2: float = 1.0
    mode: str = "decode"     # "decode" or "prefill"
    residual: bool = False   # stack glue between layers
    tag_recipe: str = "fixed"
    router_scale: int = 1    # exact power-of-two scaling of Wg
    shared_mean_x: bool = False
    note: str = ""
    fixed_tags: tuple = field(default_factory=tuple)

    # ---- sizes -----------------------------------------------------------
    def expert_params(self) -> int:
        return 3 * self.d_model * self.d_ff


TINY = Workload(
    name="tiny_d256_f512_e8_t4", seed=0, d_model=256, d_ff=512, n_experts=8,
    top_k=2, n_tokens=4, t1=1.0, t2=1.0,
    fixed_tags=(TAG_FP16,) * 4 + (TAG_INT4,) * 2 + (TAG_INT2,) * 2,
    note="experts 0-3 fp16, 4-5 int4, 6-7 int2")

MIXTRAL_T1 = Workload(
    name="mixtral_layer_decode_t1", seed=1, d_model=4096, d_ff=14336,
    n_experts=8, top_k=2, n_tokens=1, t1=0.7, t2=1.0,
    fixed_tags=(TAG_FP16,) * 4 + (TAG_MISS_INT4,) * 4,
    note="experts 0-3 cached fp16; 4-7 miss -> int4 when gate < 0.3 "
         "(Eq. 2 with T1 = 0.7, T2 = 1 at top-2)")

MIXTRAL_T8_SKEW = Workload(
    name="mixtral_layer_decode_t8_skew", seed=2, d_model=4096, d_ff=14336,
    n_experts=8, top_k=2, n_tokens=8, t1=1.0, t2=1.0, tag_recipe="431",
    router_scale=4, shared_mean_x=True,
    note="seeded fp16:int4:int2 = 4:3:1 map; Wg x4 and shared-mean tokens")

PHI_STACK = Workload(
    name="phi_moe_stack32_decode_t4", seed=3, d_model=4096, d_ff=6400,
    n_experts=16, top_k=2, n_tokens=4, n_layers=32, t1=1.0, t2=1.0,
    residual=True, tag_recipe="half",
    note="per layer 8 fp16 / 8 int4 experts; 32 layers, residual glue")

MIXTRAL_PREFILL = Workload(
    name="mixtral_stack32_prefill_t512", seed=4, d_model=4096, d_ff=14336,
    n_experts=8, top_k=2, n_tokens=512, n_layers=32, t1=1.0, t2=1.0,
    mode="prefill", residual=True, tag_recipe="431",
    note="per-layer seeded 4:3:1 map; MFMA grouped GEMM")

# int8 model (Section 4.1: int2 copies replace int8 experts), thresholds as
# quoted for Mixtral in Section 3.2: every Eq. 2 outcome (int8, int2, skip)
MIXTRAL_INT8_T1 = Workload(
    name="mixtral_int8_layer_decode_t1", seed=5, d_model=4096, d_ff=14336,
    n_experts=8, top_k=2, n_tokens=1, t1=0.6, t2=0.9,
    fixed_tags=(TAG_INT8,) * 4 + (TAG_MISS_INT8_INT2,) * 4,
    note="int8 model: experts 0-3 cached int8; 4-7 miss -> int8 / int2 / skip "
         "(Eq. 2 with T1 = 0.6, T2 = 0.9)")

ALL = [TINY, MIXTRAL_T1, MIXTRAL_T8_SKEW, PHI_STACK, MIXTRAL_PREFILL, MIXTRAL_INT8_T1]
BY_NAME = {w.name: w for w in ALL}


def seeded_permutation(seed: int, layer: int, n: int) -> np.ndarray:
    """Permutation of range(n) from the keyed stream (stable argsort of n
    16-bit draws)."""
    u = uniform_u16(tensor_key(seed, layer, TENSOR_TAGS, 0), n)
    return np.argsort(u, kind="stable")


def layer_tags(wl: Workload, layer: int) -> np.ndarray:
    """Per-expert tag of one layer."""
    E = wl.n_experts
    if wl.tag_recipe == "fixed":
        return np.array(wl.fixed_tags, dtype=np.int32)
    perm = seeded_permutation(wl.seed, layer, E)
    tags = np.empty(E, dtype=np.int32)
    if wl.tag_recipe == "431":
        n16, n4 = E * 4 // 8, E * 3 // 8
        tags[perm[:n16]] = TAG_FP16
        tags[perm[n16:n16 + n4]] = TAG_INT4
        tags[perm[n16 + n4:]] = TAG_INT2
    elif wl.tag_recipe == "half":
        tags[perm[:E // 2]] = TAG_FP16
        tags[perm[E // 2:]] = TAG_INT4
    else:
        raise ValueError(wl.tag_recipe)
    return tags


def hidden_states(wl: Workload, n_tokens: int | None = None,
                  stream: int = 0) -> np.ndarray:
    """fp16 [T, d] hidden states of the first layer.  ``stream`` selects an
    independent batch of tokens (used to vary tokens across bench steps)."""
    T = wl.n_tokens if n_tokens is None else n_tokens
    d = wl.d_model
    z = normal_fp16(wl.seed, 1000 + stream, TENSOR_X, 0, (T, d), X_STD)
    if not wl.shared_mean_x:
        return z
    # skewed routing: tokens share a common random direction m,
    # x_t = fp16((z_t + m) / sqrt(2)), computed in float32 on the host.
    m = normal_fp16(wl.seed, 1000 + stream, TENSOR_XMEAN, 0, (1, d), X_STD)
    v = (z.astype(np.float32) + m.astype(np.float32)) * np.float32(1 / np.sqrt(2))
    return v.astype(np.float16)


def router_weight(wl: Workload, layer: int) -> np.ndarray:
    """fp16 [E, d] gating weights (times an exact power of two for the skewed
    workload)."""
    wg = normal_fp16(wl.seed, layer, TENSOR_WG, 0, (wl.n_experts, wl.d_model),
                     W_STD)
    if wl.router_scale != 1:
        wg = (wg * np.float16(wl.router_scale)).astype(np.float16)
    return wg


def expert_weight(wl: Workload, layer: int, expert: int, which: str,
                  row0: int = 0, row1: int | None = None) -> np.ndarray:
    """fp16 rows [row0, row1) of W1 / W3 ([d_ff, d_model]) or W2
    ([d_model, d_ff]) of one expert."""
    tid = {"w1": TENSOR_W1, "w3": TENSOR_W3, "w2": TENSOR_W2}[which]
    rows, cols = ((wl.d_ff, wl.d_model) if which in ("w1", "w3")
                  else (wl.d_model, wl.d_ff))
    row1 = rows if row1 is None else row1
    return normal_fp16(wl.seed, layer, tid, expert, (row1 - row0, cols),
                       W_STD, start=row0 * cols)


def expert_tensor_key(wl: Workload, layer: int, expert: int, which: str) -> int:
    tid = {"w1": TENSOR_W1, "w3": TENSOR_W3, "w2": TENSOR_W2}[which]
    return tensor_key(wl.seed, layer, tid, expert)
