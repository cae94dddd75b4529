"""MI355X (gfx950) per-operator decoder-layer forward: RMSNorm, linear, SwiGLU,
ragged causal GQA prefill attention and paged decode attention, plus RoPE, the
paged KV-cache write and residual-add RMSNorm, and the mixture-of-experts FFN
(top-k routing, fused expert MLPs), as hand-written HIP kernels
behind the C ABI in include/opscale.h.  This package holds the HIP sources
(csrc/), their build script, the ctypes binding, a layer chained from the
entry points (layer), the operator profiler (profiler) and spatial sharing
over CU-masked streams (spatial)."""
from ._lib import (  # noqa: F401
    OpscaleError, Timing, Profile, OpDesc, load, LIB_PATH, EXPORTS,
    opscale_version, opscale_rmsnorm, opscale_linear, opscale_linear_workspace_size, opscale_swiglu,
    opscale_attn_prefill, opscale_set_tuning, opscale_get_tuning,
    opscale_rope, opscale_reshape_and_cache, opscale_add_rmsnorm,
    opscale_attn_decode_workspace_size, opscale_attn_decode, opscale_op_profile,
    opscale_attn_decode_noalloc, opscale_attn_decode_noalloc_max_bytes,
    desc_rmsnorm, desc_linear, desc_swiglu, desc_attn_prefill, desc_attn_decode,
    desc_rope, desc_reshape_and_cache, desc_add_rmsnorm,
    opscale_moe_topk, opscale_fused_moe_workspace_size, opscale_fused_moe, desc_fused_moe,
    Corun, opscale_cu_layout, opscale_cu_mask_build, opscale_cu_stream_create, opscale_cu_stream_destroy,
    opscale_cu_stream_mask, opscale_cu_probe, opscale_probe_mfma, opscale_probe_hbm, opscale_corun_profile,
    OPSCALE_OK, OPSCALE_ERR_INVALID_ARG, OPSCALE_ERR_UNSUPPORTED, OPSCALE_ERR_WORKSPACE,
    OPSCALE_ERR_HIP, OPSCALE_F32, OPSCALE_BF16,
    TUNE_AUTO, TUNE_GEMM_TILE, TUNE_GEMM_SKINNY, TUNE_GEMM_SPLITK, TUNE_GEMM_TAIL, TUNE_SKINNY_NG,
    TUNE_PREFILL_SCHEDULE, TUNE_MOE_FUSE, TUNE_GEMM_DECODE,
)
