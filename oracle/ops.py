"""fp64 definitions of the decoder-layer operators (test infrastructure only).

The paper (Section 2.1, "Cross-Dimension Analysis" and the sensitivity study;
Appendix C, "Dataflow Characteristics") treats a decoder layer as a dataflow of
separately profiled operators: RMS Norm, QKV Linear, attention, the MLP linears
and the fused SiLU-multiply activation.  It does not print their formulas, so
each function below is the standard definition of the named operator, written
out in fp64.  The readings taken where the paper is silent are listed in the
module-level READINGS dict and repeated in the design notes.

All arrays are converted to float64 on entry.  Outputs are float64 and are never
rounded to a narrower type.
"""
from __future__ import annotations

import numpy as np

READINGS = {
    "rmsnorm": "y = x / sqrt(mean(x^2) + eps) * w; eps inside the root; gain w multiplies "
               "(not 1+w).",
    "linear": "y = x W^T (+ b), W stored [N, K] row-major.",
    "swiglu": "input [M, 2F]: first F columns are the gate, last F the up projection; "
              "out = silu(gate) * up, silu(z) = z / (1 + exp(-z)).",
    "gqa": "query head h reads KV head h // (Hq / Hkv) (contiguous groups).",
    "causal": "within one prompt, key j is visible to query i iff j <= i; prompts do not "
              "see each other.",
    "scale": "scores are scale * q.k with scale passed in (1/sqrt(D) in the workloads).",
    "decode": "one query per sequence attends to all context_lens[b] cached keys; the new "
              "token's K/V is already in the cache; context_len 0 gives a zero output.",
    "paged": "cached key j of sequence b lives in physical block block_table[b, j // bs] "
             "at slot j % bs; cache layout [num_blocks, bs, Hkv, D].",
    "rope": "rotate-half rotary embedding (Llama family): pair (i, i + D/2), inverse frequency "
            "theta^(-2i/D), angle = position * frequency, no frequency scaling; applied to the "
            "query and key heads before attention and before the cache write.",
    "cache_write": "token t is written to physical slot slot_mapping[t] = block * bs + offset; a "
                   "slot outside [0, num_blocks * bs) is skipped (padding).",
    "residual": "r = x + residual feeds RMS Norm; r is also the residual of the next operator pair "
                "(the norm of the unrounded sum).",
}


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------- RMS Norm ---
def rmsnorm(x, w, eps: float) -> np.ndarray:
    """RMS Norm (Section 2.1: the memory-heavy, compute-light operator).

    y[m, j] = x[m, j] / sqrt((1/H) * sum_j x[m, j]^2 + eps) * w[j]
    """
    x = _f64(x)
    w = _f64(w)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * w


# ------------------------------------------------------------------ Linear ---
def linear(x, W, b=None) -> np.ndarray:
    """Linear projection (Section 2.1: QKV Linear, wide projections, MLP).

    y[m, n] = sum_k x[m, k] * W[n, k] (+ b[n]), with W stored [N, K].
    """
    y = np.matmul(_f64(x), _f64(W).T)
    if b is not None:
        y = y + _f64(b)
    return y


# ---------------------------------------------------------- SiLU-and-mul ---
def silu(z) -> np.ndarray:
    """silu(z) = z * sigmoid(z) = z / (1 + exp(-z))."""
    z = _f64(z)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu(u) -> np.ndarray:
    """Fused act_and_mul / "SiLu Mul" (Section 2.1 memory study; Appendix C).

    u is the merged gate-up projection output [M, 2F]; out = silu(u[:, :F]) * u[:, F:].
    """
    u = _f64(u)
    F = u.shape[-1] // 2
    return silu(u[..., :F]) * u[..., F:]


# ----------------------------------------------------------------- softmax ---
def softmax(s, axis: int = -1) -> np.ndarray:
    """Row softmax exp(s - max s) / sum exp(s - max s) in fp64."""
    s = _f64(s)
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


# -------------------------------------------------------- prefill attention --
def _kv_head(h: int, n_q_heads: int, n_kv_heads: int) -> int:
    return h // (n_q_heads // n_kv_heads)


def attn_prefill(q, k, v, cu_seqlens, scale: float, causal: bool = True) -> np.ndarray:
    """Self-attention over a ragged batch of prompts (Section 2.1: quadratic in
    sequence length; FlashAttention gives the same result without storing the
    score matrix; grouped-query attention as in the Table 3 models).

    q: [T, Hq, D]; k, v: [T, Hkv, D]; cu_seqlens: [B+1] prompt offsets.
    For prompt b, query i and head h (KV head g = h // (Hq/Hkv)):
        s_j = scale * q[c_b+i, h] . k[c_b+j, g]   for visible j
        o[c_b+i, h] = sum_j softmax(s)_j * v[c_b+j, g]
    The full score matrix of each (prompt, head) is materialized.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    out = np.zeros((T, Hq, D), np.float64)
    cu = np.asarray(cu_seqlens, np.int64)
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        if L == 0:
            continue
        visible = np.tril(np.ones((L, L), bool)) if causal else np.ones((L, L), bool)
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            s = scale * (q[s0:s1, h, :] @ k[s0:s1, g, :].T)
            s = np.where(visible, s, -np.inf)
            p = softmax(s, axis=-1)
            out[s0:s1, h, :] = p @ v[s0:s1, g, :]
    return out


def attn_prefill_rows(q, k, v, cu_seqlens, rows, scale: float, causal: bool = True):
    """The same definition evaluated only at the (token, head) pairs in `rows`.

    Returns an array [len(rows), D].  Used for sampled parity at full size.
    """
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    Hq = q.shape[1]
    Hkv = k.shape[1]
    cu = np.asarray(cu_seqlens, np.int64)
    out = np.zeros((len(rows), q.shape[2]), np.float64)
    for r, (t, h) in enumerate(rows):
        b = int(np.searchsorted(cu, t, side="right") - 1)
        s0, s1 = int(cu[b]), int(cu[b + 1])
        last = t if causal else s1 - 1
        g = _kv_head(int(h), Hq, Hkv)
        kk = _f64(k[s0:last + 1, g, :])
        vv = _f64(v[s0:last + 1, g, :])
        s = scale * (kk @ _f64(q[t, h, :]))
        p = softmax(s)
        out[r] = p @ vv
    return out


# --------------------------------------------------------- decode attention --
def gather_paged(cache, block_table_row, n: int) -> np.ndarray:
    """Keys (or values) 0..n-1 of one sequence from a paged cache
    [num_blocks, bs, Hkv, D]: row j = cache[block_table_row[j // bs], j % bs]."""
    bs = cache.shape[1]
    j = np.arange(n)
    return np.asarray(cache)[np.asarray(block_table_row)[j // bs], j % bs]


def attn_decode(q, k_cache, v_cache, block_table, context_lens, scale: float) -> np.ndarray:
    """One-token decode attention over a paged KV cache (Section 2.1 decode
    phase; Appendix E: decode is memory-bound; PagedAttention in the serving
    engine of Section 5).

    q: [B, Hq, D]; k_cache, v_cache: [num_blocks, bs, Hkv, D];
    block_table: [B, max_blocks]; context_lens: [B].
    o[b, h] = sum_{j < n_b} softmax_j(scale * q[b, h] . K_b[j, g]) V_b[j, g].
    """
    q = _f64(q)
    B, Hq, D = q.shape
    Hkv = k_cache.shape[2]
    out = np.zeros((B, Hq, D), np.float64)
    for b in range(B):
        n = int(context_lens[b])
        if n == 0:
            continue
        K = _f64(gather_paged(k_cache, block_table[b], n))  # [n, Hkv, D]
        V = _f64(gather_paged(v_cache, block_table[b], n))
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            p = softmax(scale * (K[:, g, :] @ q[b, h, :]))
            out[b, h] = p @ V[:, g, :]
    return out


# -------------------------------------------------------- rotary embedding ---
def rope(x, positions, theta: float) -> np.ndarray:
    """Rotary position embedding of query or key heads (the RoPE attention
    operator that Section 5.6 lists among the operators shared by Llama-family
    generations).  The paper prints no formula; this is the rotate-half form:
    for pair i < D/2, inverse frequency f_i = theta^(-2i/D), angle a = p * f_i,
        out[i]       = x[i] cos a - x[i + D/2] sin a
        out[i + D/2] = x[i + D/2] cos a + x[i] sin a.
    x: [T, H, D]; positions: [T] integer position of each token in its sequence.
    """
    x = _f64(x)
    D = x.shape[-1]
    half = D // 2
    inv_freq = float(theta) ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(positions, np.float64)[:, None] * inv_freq[None, :]  # [T, D/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


# ------------------------------------------------------------ KV cache write --
def reshape_and_cache(k, v, k_cache, v_cache, slot_mapping):
    """Write the K/V rows of new tokens into the paged cache (the
    reshape_and_cache operator of Section 2.1's memory study).  Token t goes to
    physical slot slot_mapping[t]: block slot // bs, offset slot % bs; a slot
    outside [0, num_blocks * bs) is skipped.
    k, v: [T, Hkv, D]; caches: [num_blocks, bs, Hkv, D].  Returns updated
    copies of both caches (fp64)."""
    kc = _f64(k_cache).copy()
    vc = _f64(v_cache).copy()
    nb, bs = kc.shape[0], kc.shape[1]
    k, v = _f64(k), _f64(v)
    for t, slot in enumerate(np.asarray(slot_mapping, np.int64)):
        if 0 <= slot < nb * bs:
            kc[slot // bs, slot % bs] = k[t]
            vc[slot // bs, slot % bs] = v[t]
    return kc, vc


# ------------------------------------------------------- residual + RMS Norm --
def add_rmsnorm(x, residual, w, eps: float):
    """Residual add followed by RMS Norm, the pattern each norm of a decoder
    layer sees.  r = x + residual; y = rmsnorm(r, w, eps).  Returns (y, r); r
    is the residual carried to the next norm."""
    r = _f64(x) + _f64(residual)
    return rmsnorm(r, w, eps), r


# ----------------------------------------------------- whole decoder layer ---
def decoder_layer_forward(x, residual, p, positions, cu_seqlens, n_q_heads, n_kv_heads, head_dim, eps,
                          theta, k_cache, v_cache, slot_mapping):
    """One decoder layer over a ragged prefill batch with every operator of its
    dataflow (Section 2.2): residual + norm -> QKV -> RoPE on q and k -> cache
    write of k and v -> causal attention -> O -> residual + norm -> gate-up ->
    SiLU-mul -> down.  residual None means x is the layer's first input (the
    residual is x itself).  Returns every intermediate, the layer output y, the
    residual carried to the next layer and the updated caches (all fp64)."""
    T, D = x.shape[0], head_dim
    if residual is None:
        h1, r1 = rmsnorm(x, p["w_norm1"], eps), _f64(x)
    else:
        h1, r1 = add_rmsnorm(x, residual, p["w_norm1"], eps)
    qkv = linear(h1, p["w_qkv"])
    q = rope(qkv[:, : n_q_heads * D].reshape(T, n_q_heads, D), positions, theta)
    k = rope(qkv[:, n_q_heads * D:(n_q_heads + n_kv_heads) * D].reshape(T, n_kv_heads, D), positions, theta)
    v = qkv[:, (n_q_heads + n_kv_heads) * D:].reshape(T, n_kv_heads, D)
    kc, vc = reshape_and_cache(k, v, k_cache, v_cache, slot_mapping)
    a = attn_prefill(q, k, v, cu_seqlens, 1.0 / np.sqrt(D), causal=True)
    o = linear(a.reshape(T, n_q_heads * D), p["w_o"])
    h2, r2 = add_rmsnorm(o, r1, p["w_norm2"], eps)
    gu = linear(h2, p["w_gate_up"])
    act = swiglu(gu)
    y = linear(act, p["w_down"])
    return {"h1": h1, "r1": r1, "qkv": qkv, "q": q, "k": k, "v": v, "attn": a, "o": o, "h2": h2, "r2": r2,
            "gate_up": gu, "act": act, "y": y, "k_cache": kc, "v_cache": vc}


def decoder_layer_decode(x, residual, p, context_lens, block_table, n_q_heads, n_kv_heads, head_dim, eps,
                         theta, k_cache, v_cache):
    """One decode step of the same layer for B sequences with one new token each
    (Section 2.1's 1-token decode phase; Appendix E): the new token of sequence
    b sits at position context_lens[b] - 1, its k and v are written to that
    position's cache slot before decode attention reads the whole context."""
    B, D = x.shape[0], head_dim
    ctx = np.asarray(context_lens, np.int64)
    bt = np.asarray(block_table, np.int64)
    bs = np.asarray(k_cache).shape[1]
    pos = ctx - 1
    slots = np.array([bt[b, pos[b] // bs] * bs + pos[b] % bs if pos[b] >= 0 else -1 for b in range(B)], np.int64)
    if residual is None:
        h1, r1 = rmsnorm(x, p["w_norm1"], eps), _f64(x)
    else:
        h1, r1 = add_rmsnorm(x, residual, p["w_norm1"], eps)
    qkv = linear(h1, p["w_qkv"])
    q = rope(qkv[:, : n_q_heads * D].reshape(B, n_q_heads, D), pos, theta)
    k = rope(qkv[:, n_q_heads * D:(n_q_heads + n_kv_heads) * D].reshape(B, n_kv_heads, D), pos, theta)
    v = qkv[:, (n_q_heads + n_kv_heads) * D:].reshape(B, n_kv_heads, D)
    kc, vc = reshape_and_cache(k, v, k_cache, v_cache, slots)
    a = attn_decode(q, kc, vc, bt, ctx, 1.0 / np.sqrt(D))
    o = linear(a.reshape(B, n_q_heads * D), p["w_o"])
    h2, r2 = add_rmsnorm(o, r1, p["w_norm2"], eps)
    gu = linear(h2, p["w_gate_up"])
    act = swiglu(gu)
    y = linear(act, p["w_down"])
    return {"h1": h1, "r1": r1, "qkv": qkv, "q": q, "k": k, "v": v, "slots": slots, "attn": a, "o": o,
            "h2": h2, "r2": r2, "gate_up": gu, "act": act, "y": y, "k_cache": kc, "v_cache": vc}
