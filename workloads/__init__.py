"""Seeded synthetic workloads for the per-operator decoder-layer forward.

This module only draws numbers: prompt/context lengths, random tensors and paged
block tables.  It holds none of the operators' arithmetic, so both the CPU
oracle (tests) and the HIP path (tests, bench) can take their inputs from here
without sharing any of the method.

Shapes follow the Llama-style layers the paper profiles (Section 2.1, Table 3):
an 8B layer (hidden 4096, 32 query / 8 KV heads of 128, FFN 14336) and a 70B
layer (hidden 8192, 64 / 8 heads, FFN 28672).  The paper's workloads are
production traces and real weights; seeded length distributions and normal
tensors stand in for them.

Recipe (every config):
  * rng = numpy.random.default_rng(seed) (seed 0 by default), lengths drawn first;
  * lognormal(median m, sigma s) means rng.lognormal(log(m), s), rounded to the
    nearest integer, then clipped;
  * integer-uniform [a, b] is inclusive on both ends;
  * tensors come from per-tensor generators default_rng([seed, tag]) so each
    operator's inputs can be drawn without drawing the others;
  * weights ~ N(0, 0.02), activations / q / k / v / KV cache ~ N(0, 1);
    the RMSNorm gain is 1 + N(0, 0.02) (a gain near zero would be degenerate);
  * bf16 inputs are drawn in fp32 and rounded to bf16 (nearest-even) once; the
    oracle then sees the rounded values exactly, upcast to fp64.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

# tags for per-tensor generators (stable: changing them changes every input)
TAG = {
    "x": 1, "w_norm": 2, "w_qkv": 3, "w_o": 4, "w_gate_up": 5, "w_down": 6,
    "q": 7, "k": 8, "v": 9, "gate_up": 10, "k_cache": 11, "v_cache": 12,
    "block_table": 13, "attn_out": 14, "ffn_act": 15, "dq": 16, "bias": 17,
    "moe_w1": 18, "moe_w2": 19, "router": 20,
}


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    dtype: str            # "f32" or "bf16"
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    eps: float = 1e-5
    mode: str = "prefill"  # "prefill" or "decode"
    block_size: int = 16   # paged KV cache (decode)
    seed: int = 0
    rope_theta: float = 500000.0  # rotary base of the Llama-3 family

    @property
    def qkv_out(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


def _lognormal_lengths(rng, n, median, sigma, lo, hi) -> np.ndarray:
    x = rng.lognormal(mean=math.log(median), sigma=sigma, size=n)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def _lognormal_until(rng, total, median, sigma, lo, hi) -> np.ndarray:
    """Draw lognormal lengths until they reach `total`; the last one is cut to
    the remainder, and a remainder below `lo` is merged into the previous one."""
    out: List[int] = []
    acc = 0
    while acc < total:
        v = int(np.clip(np.rint(rng.lognormal(math.log(median), sigma)), lo, hi))
        v = min(v, total - acc)
        if v < lo and out:
            out[-1] += v
        else:
            out.append(v)
        acc += v
    return np.asarray(out, np.int64)


# The five workloads.  Names describe the layer and batch they model.
C1 = LayerConfig("tiny_f32_prefill", "f32", 256, 4, 4, 64, 688, rope_theta=10000.0)
C2 = LayerConfig("llama8b_prefill_ragged16", "bf16", 4096, 32, 8, 128, 14336)
C3 = LayerConfig("llama8b_decode_b256", "bf16", 4096, 32, 8, 128, 14336, mode="decode")
C4 = LayerConfig("llama70b_prefill_16k", "bf16", 8192, 64, 8, 128, 28672)
C5 = LayerConfig("llama8b_bursty_longctx", "bf16", 4096, 32, 8, 128, 14336)
CONFIGS = {c.name: c for c in (C1, C2, C3, C4, C5)}


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    """The FFN of a mixture-of-experts layer (the paper's MoE models, Table 3):
    E experts of hidden H and expert width F, topk routed experts per token."""
    name: str
    hidden: int
    ffn: int
    experts: int
    topk: int
    tokens: int
    seed: int = 0


# Mixtral-8x7B: 8 experts of 14336, top-2; Qwen2-57B-A14B: 64 experts of 2560,
# top-8 (its shared expert is a dense MLP and not part of the routed operator).
# Routing is synthetic: router logits ~ N(0, 1), iid per token and expert,
# through top-k softmax with the k weights renormalized.
MOE_MIXTRAL_PREFILL = MoEConfig("mixtral8x7b_moe_prefill8871", 4096, 14336, 8, 2, 8871)
MOE_QWEN_DECODE = MoEConfig("qwen2_57b_a14b_moe_decode256", 3584, 2560, 64, 8, 256)
ORDER = [C1.name, C2.name, C3.name, C4.name, C5.name]


def seq_lengths(cfg: LayerConfig) -> np.ndarray:
    """Prompt lengths (prefill) or KV-cache context lengths (decode)."""
    rng = np.random.default_rng(cfg.seed)
    if cfg is C1 or cfg.name == C1.name:
        return np.asarray([128], np.int64)
    if cfg.name == C2.name:
        return _lognormal_lengths(rng, 16, 512, 1.0, 16, 4096)
    if cfg.name == C3.name:
        return rng.integers(128, 8192, size=256, endpoint=True).astype(np.int64)
    if cfg.name == C4.name:
        return _lognormal_until(rng, 16384, 1024, 0.8, 32, 8192)
    if cfg.name == C5.name:
        short = rng.integers(64, 1024, size=64, endpoint=True).astype(np.int64)
        return np.concatenate([np.full(4, 32768, np.int64), short])
    raise KeyError(cfg.name)


def cu_seqlens(lengths) -> np.ndarray:
    lengths = np.asarray(lengths, np.int64)
    out = np.zeros(len(lengths) + 1, np.int32)
    out[1:] = np.cumsum(lengths)
    return out


def rng_for(cfg_or_seed, tag: str) -> np.random.Generator:
    seed = cfg_or_seed.seed if isinstance(cfg_or_seed, LayerConfig) else int(cfg_or_seed)
    return np.random.default_rng([seed, TAG[tag]])


def normal(rng: np.random.Generator, shape, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """fp32 normal draws (bf16 rounding, if any, is applied by `as_dtype`)."""
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if mean != 0.0:
        a += np.float32(mean)
    return a


def as_dtype(a: np.ndarray, dtype: str):
    """Return a torch CPU tensor in the workload dtype (bf16: nearest-even)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    if dtype == "f32":
        return t
    raise ValueError(dtype)


def to_f64(t) -> np.ndarray:
    """Exact fp64 copy of a torch CPU tensor (bf16 and fp32 upcast exactly)."""
    import torch
    return t.detach().to("cpu", torch.float64).numpy()


def paged_cache_layout(context_lens, block_size: int, rng: np.random.Generator,
                       extra_blocks: int = 0):
    """Shuffled block table for a paged KV cache.

    Returns (block_table [B, max_blocks] int32 with unused entries 0,
    num_blocks).  Every sequence gets ceil(n_b / block_size) distinct physical
    blocks drawn from a random permutation, so pages of one sequence are
    scattered across the cache as they are after a long serving run.
    """
    context_lens = np.asarray(context_lens, np.int64)
    nblk = (context_lens + block_size - 1) // block_size
    total = int(nblk.sum()) + int(extra_blocks)
    perm = rng.permutation(total).astype(np.int32)
    max_blocks = int(max(1, nblk.max() if len(nblk) else 1))
    table = np.zeros((len(context_lens), max_blocks), np.int32)
    pos = 0
    for b, n in enumerate(nblk):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    return table, total


def pick_rows(rng: np.random.Generator, m: int, count: int) -> np.ndarray:
    """Sorted sample of row indices that always includes the first and last row."""
    if m <= count + 2:
        return np.arange(m, dtype=np.int64)
    r = rng.choice(m, size=count, replace=False)
    return np.unique(np.concatenate([r, [0, m - 1]])).astype(np.int64)


def device_normal(shape, seed: int, tag: str, dtype: str, std: float = 1.0, mean: float = 0.0,
                  device: str = "cuda"):
    """Seeded normal tensor drawn on the GPU with torch's Philox generator, for
    full-size workloads whose host generation would be slow.  Deterministic for
    a given (seed, tag).  The draws differ from `normal`'s; tests that need the
    values on the host copy the rows they check."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + TAG[tag])
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(mean=mean, std=std, generator=g)
    return t.to(dt)


def prefill_layer_inputs(cfg: LayerConfig, device: str = "cuda"):
    """Full-size inputs of one prefill layer on the GPU: the activation x
    [M, H], the layer weights (nn.Linear layout [out, in]) and cu_seqlens.
    Weights N(0, 0.02); norm gains 1 + N(0, 0.02); x N(0, 1)."""
    import torch
    lens = seq_lengths(cfg)
    cu = cu_seqlens(lens)
    M = int(cu[-1])
    H, F, dt, s = cfg.hidden, cfg.ffn, cfg.dtype, cfg.seed
    return {
        "lengths": lens,
        "cu_seqlens_host": cu,
        "cu_seqlens": torch.from_numpy(cu).to(device),
        "M": M,
        "x": device_normal((M, H), s, "x", dt, device=device),
        "w_norm1": device_normal((H,), s, "w_norm", dt, std=0.02, mean=1.0, device=device),
        "w_norm2": device_normal((H,), s + 1, "w_norm", dt, std=0.02, mean=1.0, device=device),
        "w_qkv": device_normal((cfg.qkv_out, H), s, "w_qkv", dt, std=0.02, device=device),
        "w_o": device_normal((H, cfg.n_q_heads * cfg.head_dim), s, "w_o", dt, std=0.02, device=device),
        "w_gate_up": device_normal((2 * F, H), s, "w_gate_up", dt, std=0.02, device=device),
        "w_down": device_normal((H, F), s, "w_down", dt, std=0.02, device=device),
    }


def decode_inputs(cfg: LayerConfig, device: str = "cuda"):
    """Full-size decode-attention inputs on the GPU: q [B, Hq, D], the paged
    K/V caches [num_blocks, block_size, Hkv, D] (N(0, 1)), a shuffled block
    table and the context lengths."""
    import torch
    ctx = seq_lengths(cfg)
    table, nb = paged_cache_layout(ctx, cfg.block_size, rng_for(cfg, "block_table"))
    B, dt, s = len(ctx), cfg.dtype, cfg.seed
    shape = (nb, cfg.block_size, cfg.n_kv_heads, cfg.head_dim)
    return {
        "context_lens_host": ctx,
        "block_table_host": table,
        "context_lens": torch.from_numpy(ctx.astype(np.int32)).to(device),
        "block_table": torch.from_numpy(table).to(device),
        "num_blocks": nb,
        "max_context_len": int(ctx.max()),
        "q": device_normal((B, cfg.n_q_heads, cfg.head_dim), s, "q", dt, device=device),
        "k_cache": device_normal(shape, s, "k_cache", dt, device=device),
        "v_cache": device_normal(shape, s, "v_cache", dt, device=device),
    }
