"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times, checked against the fp64 oracle on sampled outputs:
  * norm / SwiGLU: 256 random rows (+ first and last);
  * linears: 64 random rows (+ first and last), every output column;
  * prefill attention: 256 random (token, head) pairs, the first and last query
    of every prompt for every head, and every query of the shortest prompt;
  * decode attention: 32 random sequences (+ shortest and longest), all heads.
Inputs are seeded device draws (workloads.device_normal); the oracle reads the
rows it needs from copies of those inputs."""
import math

import numpy as np
import pytest

import oracle
import workloads as wl
from parity_util import assert_close, f64, say

pytestmark = pytest.mark.gpu

PREFILL = [wl.C2.name, wl.C4.name, wl.C5.name]


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as ops
    ops.load()
    return ops


def _rows(t, idx):
    import torch
    return f64(t[torch.as_tensor(idx, device=t.device)].cpu())


def _linear_ref(x_rows, W, chunk=8192):
    """Oracle linear on the sampled rows, W streamed in column blocks."""
    out = []
    for n0 in range(0, W.shape[0], chunk):
        out.append(oracle.linear(x_rows, f64(W[n0:n0 + chunk].cpu())))
    return np.concatenate(out, axis=1)


@pytest.mark.parametrize("name", PREFILL)
def test_prefill_layer_ops_sampled(ops, name):
    import torch
    cfg = wl.CONFIGS[name]
    say(f"full-size prefill ops: {name}")
    inp = wl.prefill_layer_inputs(cfg)
    M, H, F = inp["M"], cfg.hidden, cfg.ffn
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    rng = np.random.default_rng(123)
    rows_n = wl.pick_rows(rng, M, 256)
    rows_l = wl.pick_rows(rng, M, 64)

    # RMSNorm
    h1 = ops.opscale_rmsnorm(inp["x"], inp["w_norm1"], eps=cfg.eps)
    torch.cuda.synchronize()
    assert_close(_rows(h1, rows_n), oracle.rmsnorm(_rows(inp["x"], rows_n), f64(inp["w_norm1"].cpu()), cfg.eps),
                 cfg.dtype, f"{name} rmsnorm")
    # QKV linear (input: the GPU norm output, itself checked above)
    qkv = ops.opscale_linear(h1, inp["w_qkv"])
    torch.cuda.synchronize()
    assert_close(_rows(qkv, rows_l), _linear_ref(_rows(h1, rows_l), inp["w_qkv"]), cfg.dtype, f"{name} qkv")
    # prefill attention on views into the packed QKV output
    q = qkv[:, : Hq * D].view(M, Hq, D)
    k = qkv[:, Hq * D:(Hq + Hkv) * D].view(M, Hkv, D)
    v = qkv[:, (Hq + Hkv) * D:].view(M, Hkv, D)
    scale = 1.0 / math.sqrt(D)
    lens, cu = inp["lengths"], inp["cu_seqlens_host"]
    attn = ops.opscale_attn_prefill(q, k, v, inp["cu_seqlens"], int(lens.max()), scale, True)
    torch.cuda.synchronize()
    pairs = set()
    for t in rng.choice(M, 256, replace=False):
        pairs.add((int(t), int(rng.integers(Hq))))
    for b in range(len(lens)):
        for h in range(Hq):
            pairs.add((int(cu[b]), h))
            pairs.add((int(cu[b + 1]) - 1, h))
    bmin = int(np.argmin(lens))
    for t in range(int(cu[bmin]), int(cu[bmin + 1])):
        for h in range(Hq):
            pairs.add((t, h))
    pairs = sorted(pairs)
    qkv_h = qkv.cpu()  # inputs of the attention operator
    qh = qkv_h[:, : Hq * D].view(M, Hq, D)
    kh = qkv_h[:, Hq * D:(Hq + Hkv) * D].view(M, Hkv, D)
    vh = qkv_h[:, (Hq + Hkv) * D:].view(M, Hkv, D)
    ref = oracle.attn_prefill_rows(qh.to(torch.float64).numpy(), kh.to(torch.float64).numpy(),
                                   vh.to(torch.float64).numpy(), cu, pairs, scale, True)
    a_h = attn.cpu()
    got = np.stack([f64(a_h[t, h]) for t, h in pairs])
    assert_close(got, ref, cfg.dtype, f"{name} attn_prefill ({len(pairs)} rows)")
    # O projection
    a2 = attn.view(M, Hq * D)
    o = ops.opscale_linear(a2, inp["w_o"])
    torch.cuda.synchronize()
    assert_close(_rows(o, rows_l), _linear_ref(_rows(a2, rows_l), inp["w_o"]), cfg.dtype, f"{name} o_proj")
    del qkv, attn, a2, qkv_h
    # second norm, gate-up, SwiGLU, down
    h2 = ops.opscale_rmsnorm(o, inp["w_norm2"], eps=cfg.eps)
    gu = ops.opscale_linear(h2, inp["w_gate_up"])
    torch.cuda.synchronize()
    assert_close(_rows(gu, rows_l), _linear_ref(_rows(h2, rows_l), inp["w_gate_up"]), cfg.dtype, f"{name} gate_up")
    act = ops.opscale_swiglu(gu)
    torch.cuda.synchronize()
    assert_close(_rows(act, rows_n), oracle.swiglu(_rows(gu, rows_n)), cfg.dtype, f"{name} swiglu")
    del gu
    y = ops.opscale_linear(act, inp["w_down"])
    torch.cuda.synchronize()
    assert_close(_rows(y, rows_l), _linear_ref(_rows(act, rows_l), inp["w_down"]), cfg.dtype, f"{name} down")


def test_decode_attention_sampled(ops):
    import torch
    cfg = wl.C3
    say("full-size decode attention: " + cfg.name)
    inp = wl.decode_inputs(cfg)
    D = cfg.head_dim
    scale = 1.0 / math.sqrt(D)
    out = ops.opscale_attn_decode(inp["q"], inp["k_cache"], inp["v_cache"], inp["block_table"],
                                  inp["context_lens"], inp["max_context_len"], scale)
    torch.cuda.synchronize()
    ctx, table = inp["context_lens_host"], inp["block_table_host"]
    rng = np.random.default_rng(7)
    seqs = sorted(set(rng.choice(len(ctx), 32, replace=False).tolist()) | {int(ctx.argmin()), int(ctx.argmax())})
    for b in seqs:
        n = int(ctx[b])
        pages = table[b, : (n + cfg.block_size - 1) // cfg.block_size]
        kp = f64(inp["k_cache"][torch.as_tensor(pages, device="cuda")].cpu())
        vp = f64(inp["v_cache"][torch.as_tensor(pages, device="cuda")].cpu())
        ref = oracle.attn_decode(f64(inp["q"][b:b + 1].cpu()), kp, vp, np.arange(len(pages))[None],
                                 np.array([n]), scale)
        assert_close(f64(out[b:b + 1].cpu()), ref, cfg.dtype, f"decode seq {b} (n={n})")
    # decode-step linears at M = 256 (the same GEMM kernel at a small M)
    x = wl.device_normal((len(ctx), cfg.hidden), cfg.seed, "x", cfg.dtype)
    W = wl.device_normal((2 * cfg.ffn, cfg.hidden), cfg.seed, "w_gate_up", cfg.dtype, std=0.02)
    y = ops.opscale_linear(x, W)
    torch.cuda.synchronize()
    rows = wl.pick_rows(rng, len(ctx), 64)
    assert_close(_rows(y, rows), _linear_ref(_rows(x, rows), W), cfg.dtype, "decode gate_up M=256")
