"""Algorithmic flop and byte counts per operator call (test infrastructure only).

The paper's Operator Profiler records, per operator, its compute time T_v, its
memory M_v (weights vs. transient tensors) and its communication C_v, the
payload handed to the next operator (Section 4.2, "Operator Profiling"; Section
2.1 "Memory Sensitivity"; Appendix C "Dataflow Characteristics").  The counts
below are what each operator must compute or move at minimum: each input read
once, each output written once, weights read once, K/V read once per KV head
(the query heads of a group share it), causal attention counting only the
visible (lower-triangle) score entries.  Elementwise and exp work is not
counted as flops for the attention and activation rows.

`s` is the element size in bytes (2 for bf16, 4 for fp32).
"""
from __future__ import annotations

import numpy as np


def rmsnorm(M: int, H: int, s: int):
    flops = 4 * M * H
    nbytes = s * (2 * M * H + H)
    return flops, nbytes


def linear(M: int, N: int, K: int, s: int, bias: bool = False):
    flops = 2 * M * N * K
    nbytes = s * (M * K + N * K + M * N) + (s * N if bias else 0)
    return flops, nbytes


def swiglu(M: int, F: int, s: int):
    flops = 6 * M * F
    nbytes = 3 * s * M * F
    return flops, nbytes


def attn_prefill(lengths, Hq: int, Hkv: int, D: int, s: int, causal: bool = True):
    L = np.asarray(lengths, np.int64)
    T = int(L.sum())
    if causal:
        pairs = int(np.sum(L * (L + 1) // 2))
    else:
        pairs = int(np.sum(L * L))
    flops = 4 * D * Hq * pairs          # QK^T and PV, 2 flops per multiply-add each
    nbytes = s * (2 * T * Hq * D + 2 * T * Hkv * D)
    return flops, nbytes


def attn_decode(context_lens, Hq: int, Hkv: int, D: int, s: int, block_size: int):
    n = np.asarray(context_lens, np.int64)
    B = len(n)
    N = int(n.sum())
    nblocks = int(np.sum((n + block_size - 1) // block_size))
    flops = 4 * D * Hq * N
    nbytes = s * (2 * Hkv * D * N + 2 * B * Hq * D) + 4 * (nblocks + B)
    return flops, nbytes


def rope(T: int, Hq: int, Hkv: int, D: int, s: int):
    """Rotary embedding of q and k in place: each element read and written once
    (plus the int32 positions); 6 flops per rotated pair."""
    flops = 3 * T * (Hq + Hkv) * D
    nbytes = 2 * s * T * (Hq + Hkv) * D + 4 * T
    return flops, nbytes


def reshape_and_cache(T: int, Hkv: int, D: int, s: int):
    """KV-cache write of T tokens (all with a valid slot): k and v read once and
    written once, plus the int32 slot of each token."""
    return 0, 4 * s * T * Hkv * D + 4 * T


def add_rmsnorm(M: int, H: int, s: int):
    """Residual add + RMS Norm: x and residual read, the sum and y written."""
    flops = 5 * M * H
    nbytes = s * (4 * M * H + H)
    return flops, nbytes
