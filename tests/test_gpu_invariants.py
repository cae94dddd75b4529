"""GPU checks that tie operators together and check the timing path:
  * decode over the first n tokens == the last row of causal prefill over them
    (two different kernels, one definition);
  * relabelling physical cache blocks leaves decode unchanged;
  * a ragged batch equals its prompts run one by one;
  * bitwise run-to-run determinism of every bf16 kernel;
  * per-call timing and op_profile report the closed-form algorithmic work."""
import math

import numpy as np
import pytest

import workloads as wl
from oracle import cost
from parity_util import assert_close, cuda, f64, gen, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as ops
    ops.load()
    return ops


def test_decode_equals_last_prefill_row(ops):
    import torch
    Hq, Hkv, D, bs = 32, 8, 128, 16
    for n in (1, 37, 700):
        say(f"decode vs prefill n={n}")
        q = gen(61, "q", (n, Hq, D), "bf16")
        k = gen(61, "k", (n, Hkv, D), "bf16")
        v = gen(61, "v", (n, Hkv, D), "bf16")
        scale = 1 / math.sqrt(D)
        cu = torch.tensor([0, n], dtype=torch.int32, device="cuda")
        pre = ops.opscale_attn_prefill(cuda(q), cuda(k), cuda(v), cu, n, scale, True)
        nb = (n + bs - 1) // bs
        kc = torch.zeros(nb * bs, Hkv, D, dtype=torch.bfloat16)
        vc = torch.zeros(nb * bs, Hkv, D, dtype=torch.bfloat16)
        kc[:n], vc[:n] = k, v
        table = torch.arange(nb, dtype=torch.int32).view(1, nb)
        dec = ops.opscale_attn_decode(cuda(q[n - 1:n]), cuda(kc.view(nb, bs, Hkv, D)), cuda(vc.view(nb, bs, Hkv, D)),
                                      cuda(table), torch.tensor([n], dtype=torch.int32, device="cuda"), n, scale)
        torch.cuda.synchronize()
        assert_close(f64(dec.cpu())[0], f64(pre.cpu())[n - 1], "bf16", f"decode vs prefill n={n}")


def test_decode_block_relabel_invariance(ops):
    import torch
    ctx = np.array([300, 17, 1000])
    bs, Hkv, Hq, D = 16, 2, 8, 128
    table, nb = wl.paged_cache_layout(ctx, bs, np.random.default_rng(3))
    kc = gen(62, "k_cache", (nb, bs, Hkv, D), "bf16")
    vc = gen(62, "v_cache", (nb, bs, Hkv, D), "bf16")
    q = gen(62, "q", (3, Hq, D), "bf16")
    perm = np.random.default_rng(4).permutation(nb)
    kc2, vc2 = torch.empty_like(kc), torch.empty_like(vc)
    kc2[torch.from_numpy(perm)] = kc
    vc2[torch.from_numpy(perm)] = vc
    ctx_d = torch.from_numpy(ctx.astype(np.int32)).cuda()
    a = ops.opscale_attn_decode(cuda(q), cuda(kc), cuda(vc), cuda(torch.from_numpy(table)), ctx_d, 1000, 0.1)
    b = ops.opscale_attn_decode(cuda(q), cuda(kc2), cuda(vc2), cuda(torch.from_numpy(perm[table].astype(np.int32))),
                                ctx_d, 1000, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_prefill_batch_composition(ops):
    import torch
    lens = [300, 5, 129]
    cu = wl.cu_seqlens(lens)
    Hq, Hkv, D = 8, 2, 128
    q = cuda(gen(63, "q", (cu[-1], Hq, D), "bf16"))
    k = cuda(gen(63, "k", (cu[-1], Hkv, D), "bf16"))
    v = cuda(gen(63, "v", (cu[-1], Hkv, D), "bf16"))
    full = ops.opscale_attn_prefill(q, k, v, cuda(torch.from_numpy(cu)), 300, 0.09)
    for b in range(3):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        one = ops.opscale_attn_prefill(q[s0:s1].contiguous(), k[s0:s1].contiguous(), v[s0:s1].contiguous(),
                                       torch.tensor([0, s1 - s0], dtype=torch.int32, device="cuda"), s1 - s0, 0.09)
        torch.cuda.synchronize()
        assert torch.equal(full[s0:s1], one)


def test_bitwise_determinism(ops):
    import torch
    say("determinism")
    x = cuda(gen(64, "x", (777, 4096), "bf16"))
    w = cuda(gen(64, "w_norm", (4096,), "bf16", std=0.02, mean=1.0))
    W = cuda(gen(64, "w_qkv", (1536, 4096), "bf16", std=0.02))
    u = cuda(gen(64, "gate_up", (777, 2048), "bf16"))
    lens = [500, 277]
    cu = cuda(torch.from_numpy(wl.cu_seqlens(lens)))
    q = cuda(gen(64, "q", (777, 8, 128), "bf16"))
    kv = cuda(gen(64, "k", (777, 2, 128), "bf16"))
    ctx = np.array([777, 12])
    table, nb = wl.paged_cache_layout(ctx, 16, np.random.default_rng(5))
    kc = cuda(gen(64, "k_cache", (nb, 16, 2, 128), "bf16"))
    runs = []
    for _ in range(2):
        r = [ops.opscale_rmsnorm(x, w), ops.opscale_linear(x, W), ops.opscale_swiglu(u),
             ops.opscale_attn_prefill(q, kv, kv, cu, 500, 0.08),
             ops.opscale_attn_decode(q[:2], kc, kc, cuda(torch.from_numpy(table)),
                                     cuda(torch.from_numpy(ctx.astype(np.int32))), 777, 0.08)]
        torch.cuda.synchronize()
        runs.append(r)
    for a, b in zip(*runs):
        assert torch.equal(a, b)


def test_timing_reports_closed_form_work(ops):
    import torch
    M, H, N, F = 1000, 4096, 1024, 2048
    x = cuda(gen(65, "x", (M, H), "bf16"))
    w = cuda(gen(65, "w_norm", (H,), "bf16", std=0.02, mean=1.0))
    _, t = ops.opscale_rmsnorm(x, w, timed=True)
    assert t.elapsed_us > 0 and (t.alg_flops, t.alg_bytes) == cost.rmsnorm(M, H, 2)
    W = cuda(gen(65, "w_qkv", (N, H), "bf16", std=0.02))
    _, t = ops.opscale_linear(x, W, timed=True)
    assert t.elapsed_us > 0 and (t.alg_flops, t.alg_bytes) == cost.linear(M, N, H, 2)
    u = cuda(gen(65, "gate_up", (M, 2 * F), "bf16"))
    _, t = ops.opscale_swiglu(u, timed=True)
    assert t.elapsed_us > 0 and (t.alg_flops, t.alg_bytes) == cost.swiglu(M, F, 2)
    lens = [600, 400]
    q = cuda(gen(65, "q", (M, 8, 128), "bf16"))
    kv = cuda(gen(65, "k", (M, 2, 128), "bf16"))
    _, t = ops.opscale_attn_prefill(q, kv, kv, cuda(torch.from_numpy(wl.cu_seqlens(lens))), 600, 0.1, timed=True)
    assert t.elapsed_us > 0 and (t.alg_flops, t.alg_bytes) == cost.attn_prefill(lens, 8, 2, 128, 2)
    ctx = np.array([600, 5, 33])
    table, nb = wl.paged_cache_layout(ctx, 16, np.random.default_rng(6))
    kc = cuda(gen(65, "k_cache", (nb, 16, 2, 128), "bf16"))
    _, t = ops.opscale_attn_decode(q[:3], kc, kc, cuda(torch.from_numpy(table)),
                                   cuda(torch.from_numpy(ctx.astype(np.int32))), 600, 0.1, timed=True)
    assert t.elapsed_us > 0 and (t.alg_flops, t.alg_bytes) == cost.attn_decode(ctx, 8, 2, 128, 2, 16)


def test_op_profile(ops):
    import torch
    M, K, N = 2048, 4096, 4096
    x = cuda(gen(66, "x", (M, K), "bf16"))
    W = cuda(gen(66, "w_o", (N, K), "bf16", std=0.02))
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    p = ops.opscale_op_profile(ops.desc_linear(x, W, y), warmup=2, iters=10, flush=flush)
    d = p.as_dict()
    say(f"profile linear {M}x{N}x{K}: {d}")
    assert p.iters == 10 and 0 < p.us_min <= p.us_median <= p.us_p90
    assert (p.alg_flops, p.alg_bytes) == cost.linear(M, N, K, 2)
    assert p.bound == 0 and 0 < p.roofline_frac < 1.2
    assert p.weight_bytes == 2 * N * K and p.io_bytes == 2 * M * N
    # the profiled call computed the same result as a plain call
    ref = ops.opscale_linear(x, W)
    torch.cuda.synchronize()
    assert torch.equal(ref, y)
