"""GPU parity of the operators around attention (rotary embedding, the paged
KV-cache write, residual add + RMS Norm) and of a whole decoder layer chained
from the C-ABI calls (paper_2608_13499_amd.layer), against the fp64 oracle:
  * RoPE on packed-QKV views, fp32 and bf16, positions up to 33000; the V
    columns of the packed tensor are left bitwise untouched;
  * the cache write is a copy: bit-exact, skipped slots leave the cache as is;
  * residual + norm: both outputs (the new residual and the normalized row);
  * a layer: prefill of a ragged batch then one decode step, every
    intermediate against oracle.decoder_layer_forward / decoder_layer_decode;
  * at the 8B prefill shape (8871 tokens) the three operators on sampled rows.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from parity_util import assert_close, cuda, f64, gen, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as ops
    ops.load()
    return ops


def _packed(seed, T, Hq, Hkv, D, dtype):
    qkv = gen(seed, "q", (T, (Hq + 2 * Hkv) * D), dtype)
    return qkv


def _views(qkv, Hq, Hkv, D):
    T = qkv.shape[0]
    return (qkv[:, : Hq * D].view(T, Hq, D), qkv[:, Hq * D:(Hq + Hkv) * D].view(T, Hkv, D),
            qkv[:, (Hq + Hkv) * D:].view(T, Hkv, D))


# ------------------------------------------------------------------- RoPE ---
@pytest.mark.parametrize("dtype,T,Hq,Hkv,D,theta,maxpos", [
    ("f32", 128, 4, 4, 64, 10000.0, 128),
    ("f32", 37, 8, 2, 128, 500000.0, 33000),
    ("bf16", 300, 8, 2, 128, 500000.0, 33000),
    ("bf16", 65, 4, 4, 64, 10000.0, 4096),
    ("bf16", 1, 32, 8, 128, 500000.0, 8191),
])
def test_rope(ops, dtype, T, Hq, Hkv, D, theta, maxpos):
    import torch
    say(f"rope {dtype} T={T} Hq={Hq} Hkv={Hkv} D={D} theta={theta} maxpos={maxpos}")
    qkv = _packed(31, T, Hq, Hkv, D, dtype)
    pos = wl.rng_for(31, "block_table").integers(0, maxpos, T).astype(np.int32)
    pos[0] = 0
    qd = cuda(qkv)
    q, k, v = _views(qd, Hq, Hkv, D)
    ops.opscale_rope(q, k, cuda(torch.from_numpy(pos)), theta)
    torch.cuda.synchronize()
    got = qd.cpu()
    qh, kh, vh = _views(qkv, Hq, Hkv, D)
    gq, gk, gv = _views(got, Hq, Hkv, D)
    assert_close(f64(gq), oracle.rope(f64(qh), pos, theta), dtype, "rope q")
    assert_close(f64(gk), oracle.rope(f64(kh), pos, theta), dtype, "rope k")
    assert torch.equal(gv, vh), "rope touched the V columns"
    assert torch.equal(got[0], qkv[0]), "position 0 must be the identity"


# ------------------------------------------------------ KV-cache write ---
@pytest.mark.parametrize("dtype,T,Hkv,D,bs,nb", [("bf16", 300, 8, 128, 16, 40), ("f32", 50, 2, 64, 1, 80),
                                                 ("bf16", 1, 1, 64, 256, 2)])
def test_reshape_and_cache(ops, dtype, T, Hkv, D, bs, nb):
    import torch
    say(f"reshape_and_cache {dtype} T={T} Hkv={Hkv} D={D} bs={bs} nb={nb}")
    Hq = Hkv
    qkv = _packed(32, T, Hq, Hkv, D, dtype)
    rng = wl.rng_for(32, "block_table")
    slots = rng.permutation(nb * bs)[:T].astype(np.int32)
    if T > 2:
        slots[1], slots[2] = -1, nb * bs  # padding: skipped
    kc0 = gen(32, "k_cache", (nb, bs, Hkv, D), dtype)
    vc0 = gen(32, "v_cache", (nb, bs, Hkv, D), dtype)
    kc, vc = cuda(kc0), cuda(vc0)
    qd = cuda(qkv)
    _, k, v = _views(qd, Hq, Hkv, D)
    ops.opscale_reshape_and_cache(k, v, kc, vc, cuda(torch.from_numpy(slots)))
    torch.cuda.synchronize()
    _, kh, vh = _views(qkv, Hq, Hkv, D)
    rk, rv = oracle.reshape_and_cache(f64(kh), f64(vh), f64(kc0), f64(vc0), slots)
    np.testing.assert_array_equal(f64(kc.cpu()), rk)
    np.testing.assert_array_equal(f64(vc.cpu()), rv)


# ------------------------------------------------- residual + RMS Norm ---
@pytest.mark.parametrize("dtype,M,H,inplace", [("f32", 128, 256, False), ("bf16", 33, 4096, False),
                                               ("bf16", 1000, 8192, True), ("bf16", 1, 512, False),
                                               ("f32", 7, 4096, True)])
def test_add_rmsnorm(ops, dtype, M, H, inplace):
    import torch
    say(f"add_rmsnorm {dtype} M={M} H={H} inplace={inplace}")
    x = gen(33, "x", (M, H), dtype)
    r = gen(33, "attn_out", (M, H), dtype)
    w = gen(33, "w_norm", (H,), dtype, std=0.02, mean=1.0)
    xd, rd, wd = cuda(x), cuda(r), cuda(w)
    y = ops.opscale_add_rmsnorm(xd, rd, wd, y=xd if inplace else None, eps=1e-5)
    torch.cuda.synchronize()
    ry, rr = oracle.add_rmsnorm(f64(x), f64(r), f64(w), 1e-5)
    assert_close(f64(rd.cpu()), rr, dtype, "add_rmsnorm residual")
    assert_close(f64(y.cpu()), ry, dtype, "add_rmsnorm y")


# ----------------------------------------------------------- a whole layer ---
def _layer_weights(seed, shape, dtype):
    H, Hq, Hkv, D, F = shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn
    return {
        "w_norm1": gen(seed, "w_norm", (H,), dtype, std=0.02, mean=1.0),
        "w_qkv": gen(seed, "w_qkv", ((Hq + 2 * Hkv) * D, H), dtype, std=0.02),
        "w_o": gen(seed, "w_o", (H, Hq * D), dtype, std=0.02),
        "w_norm2": gen(seed, "bias", (H,), dtype, std=0.02, mean=1.0),
        "w_gate_up": gen(seed, "w_gate_up", (2 * F, H), dtype, std=0.02),
        "w_down": gen(seed, "w_down", (H, F), dtype, std=0.02),
    }


@pytest.mark.parametrize("dtype,H,Hq,Hkv,D,F,lens,bs,theta,first", [
    ("f32", 256, 4, 4, 64, 688, [128], 16, 10000.0, True),           # the tiny fp32 layer
    ("f32", 256, 4, 2, 64, 512, [33, 70, 1], 16, 10000.0, False),
    ("bf16", 512, 8, 2, 128, 1024, [200, 31, 97, 5], 16, 500000.0, False),
    ("bf16", 256, 4, 4, 64, 512, [64, 130], 1, 500000.0, True),
])
def test_layer_prefill_then_decode(ops, dtype, H, Hq, Hkv, D, F, lens, bs, theta, first):
    import torch
    from paper_2608_13499_amd.layer import LayerShape, decode_layer, prefill_layer
    say(f"layer {dtype} H={H} Hq={Hq} Hkv={Hkv} D={D} F={F} lens={lens} bs={bs} first={first}")
    shape = LayerShape(H, Hq, Hkv, D, F, 1e-5, theta)
    w = _layer_weights(34, shape, dtype)
    wd = {k_: cuda(v_) for k_, v_ in w.items()}
    wh = {k_: f64(v_) for k_, v_ in w.items()}
    lens = np.asarray(lens)
    T, B = int(lens.sum()), len(lens)
    cu = wl.cu_seqlens(lens)
    # a cache with room for every prompt plus one decoded token, pages shuffled
    table, nb = wl.paged_cache_layout(lens + 1, bs, wl.rng_for(34, "block_table"), extra_blocks=2)
    pos = np.concatenate([np.arange(L) for L in lens]).astype(np.int32)
    slots = np.concatenate([[table[b, j // bs] * bs + j % bs for j in range(L)] for b, L in enumerate(lens)]).astype(np.int32)
    kc0 = gen(34, "k_cache", (nb, bs, Hkv, D), dtype)
    vc0 = gen(34, "v_cache", (nb, bs, Hkv, D), dtype)
    x = gen(34, "x", (T, H), dtype)
    res = None if first else gen(34, "attn_out", (T, H), dtype)
    kc, vc = cuda(kc0), cuda(vc0)
    out = prefill_layer(shape, wd, cuda(x), None if first else cuda(res), cuda(torch.from_numpy(pos)),
                        cuda(torch.from_numpy(cu.astype(np.int32))), int(lens.max()), kc, vc,
                        cuda(torch.from_numpy(slots)))
    torch.cuda.synchronize()
    ref = oracle.decoder_layer_forward(f64(x), None if first else f64(res), wh, pos, cu, Hq, Hkv, D, 1e-5, theta,
                                       f64(kc0), f64(vc0), slots)
    q_g, k_g, _ = _views(out["qkv"].cpu(), Hq, Hkv, D)
    for name, got, want in (("h1", out["h1"], ref["h1"]), ("q (rotated)", q_g, ref["q"]), ("k (rotated)", k_g, ref["k"]),
                            ("attn", out["attn"], ref["attn"]), ("o", out["o"], ref["o"]),
                            ("h2", out["h2"], ref["h2"]), ("residual", out["residual"], ref["r2"]),
                            ("act", out["act"], ref["act"]), ("y", out["y"], ref["y"])):
        assert_close(f64(got.cpu() if hasattr(got, "cpu") else got), want, dtype, f"prefill layer {name}")
    assert_close(f64(kc.cpu()), ref["k_cache"], dtype, "prefill layer k_cache")
    assert_close(f64(vc.cpu()), ref["v_cache"], dtype, "prefill layer v_cache")

    # one decode step: token L of every sequence, on the cache the GPU prefill wrote
    ctx = (lens + 1).astype(np.int32)
    dpos = (ctx - 1).astype(np.int32)
    dslots = np.array([table[b, p // bs] * bs + p % bs for b, p in enumerate(dpos)], np.int32)
    xd = gen(35, "x", (B, H), dtype)
    rd = gen(35, "attn_out", (B, H), dtype)
    kc_before, vc_before = kc.cpu(), vc.cpu()
    dout = decode_layer(shape, wd, cuda(xd), cuda(rd), cuda(torch.from_numpy(dpos)), cuda(torch.from_numpy(dslots)),
                        kc, vc, cuda(torch.from_numpy(table)), cuda(torch.from_numpy(ctx)), int(ctx.max()))
    torch.cuda.synchronize()
    dref = oracle.decoder_layer_decode(f64(xd), f64(rd), wh, ctx, table, Hq, Hkv, D, 1e-5, theta,
                                       f64(kc_before), f64(vc_before))
    assert list(dref["slots"]) == list(dslots)
    for name in ("h1", "attn", "o", "h2", "act", "y"):
        assert_close(f64(dout[name].cpu()), dref[name], dtype, f"decode layer {name}")
    assert_close(f64(dout["residual"].cpu()), dref["r2"], dtype, "decode layer residual")


# ------------------------------------------------ full size, sampled rows ---
def test_layer_ops_full_size_sampled(ops):
    """RoPE, cache write and residual norm at the 8B prefill shape (8871
    tokens, 32 / 8 heads of 128) on sampled rows."""
    import torch
    cfg = wl.C2
    say("full-size layer ops: " + cfg.name)
    lens = wl.seq_lengths(cfg)
    cu = wl.cu_seqlens(lens)
    T, H = int(cu[-1]), cfg.hidden
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    qkv = wl.device_normal((T, (Hq + 2 * Hkv) * D), cfg.seed, "q", "bf16")
    before = qkv.clone()
    q, k, v = _views(qkv, Hq, Hkv, D)
    pos = torch.from_numpy(np.concatenate([np.arange(L) for L in lens]).astype(np.int32))
    ops.opscale_rope(q, k, cuda(pos), cfg.rope_theta)
    torch.cuda.synchronize()
    rng = np.random.default_rng(321)
    rows = wl.pick_rows(rng, T, 256)
    idx = torch.as_tensor(rows, device="cuda")
    bq, bk, _ = _views(before[idx].cpu(), Hq, Hkv, D)
    gq, gk, _ = _views(qkv[idx].cpu(), Hq, Hkv, D)
    assert_close(f64(gq), oracle.rope(f64(bq), pos.numpy()[rows], cfg.rope_theta), "bf16", "rope q (8871 tokens)")
    assert_close(f64(gk), oracle.rope(f64(bk), pos.numpy()[rows], cfg.rope_theta), "bf16", "rope k (8871 tokens)")
    assert torch.equal(v, _views(before, Hq, Hkv, D)[2])
    # cache write of every token into a shuffled paged cache
    bs = cfg.block_size
    table, nb = wl.paged_cache_layout(lens, bs, wl.rng_for(cfg, "block_table"))
    slots = np.concatenate([[table[b, j // bs] * bs + j % bs for j in range(L)] for b, L in enumerate(lens)])
    kc = torch.zeros(nb, bs, Hkv, D, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    ops.opscale_reshape_and_cache(k, v, kc, vc, cuda(torch.from_numpy(slots.astype(np.int32))))
    torch.cuda.synchronize()
    flat_k, flat_v = kc.view(nb * bs, Hkv, D), vc.view(nb * bs, Hkv, D)
    sl = torch.as_tensor(slots, device="cuda")
    assert torch.equal(flat_k[sl], k) and torch.equal(flat_v[sl], v), "cache rows differ from k / v"
    # residual + norm over the hidden state
    x = wl.device_normal((T, H), cfg.seed, "x", "bf16")
    r = wl.device_normal((T, H), cfg.seed, "attn_out", "bf16")
    w = wl.device_normal((H,), cfg.seed, "w_norm", "bf16", std=0.02, mean=1.0)
    x_rows, r_rows = f64(x[idx].cpu()), f64(r[idx].cpu())
    y = ops.opscale_add_rmsnorm(x, r, w, eps=cfg.eps)
    torch.cuda.synchronize()
    ry, rr = oracle.add_rmsnorm(x_rows, r_rows, f64(w.cpu()), cfg.eps)
    assert_close(f64(r[idx].cpu()), rr, "bf16", "add_rmsnorm residual (8871 rows)")
    assert_close(f64(y[idx].cpu()), ry, "bf16", "add_rmsnorm y (8871 rows)")
