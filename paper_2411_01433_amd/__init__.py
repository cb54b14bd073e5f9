"""Mixed-precision MoE layer (HOBBIT, arXiv 2411.01433) for AMD MI355X.

The layer runs in the HIP library libmoe.so (C ABI: include/moe.h);
this package holds its sources (csrc/), the build script and a thin ctypes
binding.  Importing the package does not load the library; the first call
that needs it does, and raises if it has not been built.
"""
from .binding import (  # noqa: F401
    EXPORTED, LIB_PATH, MOE_EHIP, MOE_EINVAL, MOE_ENOMEM, MOE_ESTATE,
    MOE_EUNSUPPORTED, MOE_OK, PREC_HIGH, PREC_LOW, PREC_SKIP, TAG_FP16,
    TAG_INT2, TAG_INT4, TAG_MISS_INT2, TAG_MISS_INT4, LayerDesc, MoeError,
    MoeCache, MoeLayer, MoePredictor, MoeStore, lib, quantize, rmsnorm,
)
