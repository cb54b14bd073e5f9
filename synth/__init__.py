"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This package generates data only. It holds none of the MoE method's
arithmetic (no gating, no quantisation, no expert math). Both the CPU
oracle and the GPU tests/benchmarks take their inputs from here, so the
two sides see bit-identical fp16 tensors.
"""
from .gen import (  # noqa: F401
    SEED_MIX,
    tensor_key,
    normal_table,
    normal_fp16,
    uniform_u16,
    TENSOR_X,
    TENSOR_WG,
    TENSOR_W1,
    TENSOR_W3,
    TENSOR_W2,
    TENSOR_XMEAN,
    TENSOR_TAGS,
)
