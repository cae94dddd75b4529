"""A whole decoder layer chained from the C-ABI operators (no compute here:
each step is one library call; this module only allocates the intermediate
tensors and passes views).

The dataflow is the operator graph of one Llama-style layer (the paper's unit
of profiling and scaling, Section 2.2):

    [residual +] RMS Norm -> QKV linear -> RoPE(q, k) -> KV-cache write(k, v)
    -> attention (prefill: causal ragged; decode: paged) -> O linear
    -> residual + RMS Norm -> gate-up linear -> SiLU-mul -> down linear

`residual` follows the usual convention: None for the first layer (the input
is its own residual), otherwise the running residual, which the two fused
norms update in place to x + residual.  The layer returns the MLP output `y`
and the residual to pass to the next layer together with `y`.
"""
from __future__ import annotations

import dataclasses
import math

from . import _lib as L


@dataclasses.dataclass(frozen=True)
class LayerShape:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    eps: float = 1e-5
    rope_theta: float = 500000.0


def _front(shape: LayerShape, w, x, residual, stream):
    """[residual +] norm and the QKV projection; returns (qkv, residual)."""
    import torch
    if residual is None:
        residual = x.clone()
        h1 = L.opscale_rmsnorm(x, w["w_norm1"], eps=shape.eps, stream=stream)
    else:
        h1 = torch.empty_like(x)
        L.opscale_add_rmsnorm(x, residual, w["w_norm1"], y=h1, eps=shape.eps, stream=stream)
    qkv = L.opscale_linear(h1, w["w_qkv"], stream=stream)
    return h1, qkv, residual


def _split(shape: LayerShape, qkv):
    T = qkv.shape[0]
    Hq, Hkv, D = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    q = qkv[:, : Hq * D].view(T, Hq, D)
    k = qkv[:, Hq * D:(Hq + Hkv) * D].view(T, Hkv, D)
    v = qkv[:, (Hq + Hkv) * D:].view(T, Hkv, D)
    return q, k, v


def _back(shape: LayerShape, w, attn, residual, stream):
    import torch
    T = attn.shape[0]
    o = L.opscale_linear(attn.view(T, -1), w["w_o"], stream=stream)
    h2 = torch.empty_like(o)
    L.opscale_add_rmsnorm(o, residual, w["w_norm2"], y=h2, eps=shape.eps, stream=stream)
    gu = L.opscale_linear(h2, w["w_gate_up"], stream=stream)
    act = L.opscale_swiglu(gu, stream=stream)
    y = L.opscale_linear(act, w["w_down"], stream=stream)
    return {"o": o, "h2": h2, "gate_up": gu, "act": act, "y": y}


def prefill_layer(shape: LayerShape, w, x, residual, positions, cu_seqlens, max_seqlen: int, k_cache, v_cache,
                  slot_mapping, stream=None):
    """One layer over a ragged prefill batch x [T, H].  positions / slot_mapping:
    int32 [T] on the GPU (position of each token in its prompt, cache slot of
    each token); cu_seqlens int32 [B + 1]."""
    h1, qkv, residual = _front(shape, w, x, residual, stream)
    q, k, v = _split(shape, qkv)
    L.opscale_rope(q, k, positions, shape.rope_theta, stream=stream)
    L.opscale_reshape_and_cache(k, v, k_cache, v_cache, slot_mapping, stream=stream)
    attn = L.opscale_attn_prefill(q, k, v, cu_seqlens, max_seqlen, 1.0 / math.sqrt(shape.head_dim), True,
                                  stream=stream)
    out = _back(shape, w, attn, residual, stream)
    out.update(h1=h1, qkv=qkv, attn=attn, residual=residual)
    return out


def decode_layer(shape: LayerShape, w, x, residual, positions, slot_mapping, k_cache, v_cache, block_table,
                 context_lens, max_context_len: int, workspace=None, stream=None):
    """One decode step of the layer for B sequences, x [B, H] (one new token
    each at positions[b] = context_lens[b] - 1, written to cache slot
    slot_mapping[b] before attention reads the whole context)."""
    h1, qkv, residual = _front(shape, w, x, residual, stream)
    q, k, v = _split(shape, qkv)
    L.opscale_rope(q, k, positions, shape.rope_theta, stream=stream)
    L.opscale_reshape_and_cache(k, v, k_cache, v_cache, slot_mapping, stream=stream)
    attn = L.opscale_attn_decode(q, k_cache, v_cache, block_table, context_lens, max_context_len,
                                 1.0 / math.sqrt(shape.head_dim), workspace=workspace, stream=stream)
    out = _back(shape, w, attn, residual, stream)
    out.update(h1=h1, qkv=qkv, attn=attn, residual=residual)
    return out
