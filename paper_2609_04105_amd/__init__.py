"""fp4attn: Direct-P full-MXFP4 attention forward for AMD MI355X (gfx950).

Thin Python binding over the C-ABI library ``libfp4attn.so`` (declared in
``include/fp4attn.h``).  Functions take PyTorch tensors only as device memory:
they check shapes, dtypes and devices, pass raw pointers and the current HIP
stream, and raise on any non-OK status.  Every step of the attention path runs
in the library's HIP kernels; there is no fallback.
"""
from ._lib import (  # noqa: F401
    FP4ATTN_BF16,
    FP4ATTN_F32,
    Fp4AttnError,
    LIB_PATH,
    abi_version,
    lib,
)
from .api import (  # noqa: F401
    attention_mxfp4,
    debug_directp_mxfp4,
    debug_mfma_stream,
    forward_bf16,
    forward_mxfp4,
    forward_options,
    quantize_mxfp4,
    quantize_mxfp8,
    quantize_qkv,
)
