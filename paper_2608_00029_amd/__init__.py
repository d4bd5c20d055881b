"""MI355X (gfx950) fused causal multi-head attention, forward and backward,
plus the fused loss head and the memory-bound operators (LayerNorm, GELU,
softmax cross entropy) of the same training step.

The compute lives in libcattn.so (HIP kernels behind the C ABI of
include/cattn.h); this package only marshals torch tensors into that ABI.
"""
from .binding import (  # noqa: F401
    CattnError, attn_bwd, attn_bwd_dkdv, attn_bwd_dq, attn_fwd, last_error_string, library_path, status_string, workspace_bytes,
    lmhead_fwd, lmhead_workspace_bytes,
    layernorm_fwd, layernorm_bwd, layernorm_bwd_workspace_bytes, gelu_fwd, gelu_bwd, sce_fwd, sce_bwd,
    CATTN_BF16, CATTN_F32, CATTN_OK, CATTN_ERR_HIP, CATTN_ERR_INVALID_ARG, CATTN_ERR_UNSUPPORTED, CATTN_BHSD, CATTN_BSHD,
)
