"""MI355X (gfx950) per-operator decoder-layer forward: RMSNorm, linear, SwiGLU,
ragged causal GQA prefill attention and paged decode attention, plus RoPE, the
paged KV-cache write and residual-add RMSNorm, as hand-written HIP kernels
behind the C ABI in include/opscale.h.  This package holds the HIP sources
(csrc/), their build script, the ctypes binding, a layer chained from the
entry points (layer) and the operator profiler (profiler)."""
from ._lib import (  # noqa: F401
    OpscaleError, Timing, Profile, OpDesc, load, LIB_PATH, EXPORTS,
    opscale_version, opscale_rmsnorm, opscale_linear, opscale_swiglu, opscale_attn_prefill,
    opscale_rope, opscale_reshape_and_cache, opscale_add_rmsnorm,
    opscale_attn_decode_workspace_size, opscale_attn_decode, opscale_op_profile,
    desc_rmsnorm, desc_linear, desc_swiglu, desc_attn_prefill, desc_attn_decode,
    desc_rope, desc_reshape_and_cache, desc_add_rmsnorm,
    OPSCALE_OK, OPSCALE_ERR_INVALID_ARG, OPSCALE_ERR_UNSUPPORTED, OPSCALE_ERR_WORKSPACE,
    OPSCALE_ERR_HIP, OPSCALE_F32, OPSCALE_BF16,
)
