"""The allocation-free decode entry point (opscale_attn_decode_noalloc), called
through the C ABI, against the workspace entry point (opscale_attn_decode) on
the same inputs and against the oracle: two calls in a row, the second with a
smaller batch, then a size beyond the library's scratch, which is rejected
before anything is enqueued."""
import math

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


def _case(seed, ctx, Hq, Hkv, D, bs):
    import torch
    ctx = np.asarray(ctx, np.int64)
    table, nb = wl.paged_cache_layout(ctx, bs, wl.rng_for(seed, "block_table"), extra_blocks=3)
    kc = gen(seed, "k_cache", (nb, bs, Hkv, D), "bf16")
    vc = gen(seed, "v_cache", (nb, bs, Hkv, D), "bf16")
    q = gen(seed, "q", (len(ctx), Hq, D), "bf16")
    dev = dict(q=cuda(q), kc=cuda(kc), vc=cuda(vc), table=cuda(torch.from_numpy(table)),
               ctx=cuda(torch.from_numpy(ctx.astype(np.int32))))
    host = dict(q=f64(q), kc=f64(kc), vc=f64(vc), table=table, ctx=ctx)
    return dev, host, int(max(1, ctx.max())), 1.0 / math.sqrt(D)


def test_noalloc_decode_matches_the_workspace_entry_point(ops):
    import torch
    rng = np.random.default_rng(7)
    cases = [
        ("200 sequences", 61, np.concatenate([rng.integers(1, 1200, 199), [0]]), 16, 4, 128, 16),
        ("3 sequences (smaller)", 62, [5, 1, 77], 8, 2, 128, 16),
    ]
    assert ops.opscale_attn_decode_noalloc_max_bytes() == 64 << 20
    for name, seed, ctx, Hq, Hkv, D, bs in cases:
        say(f"attn_decode_noalloc {name}: Hq={Hq} Hkv={Hkv} D={D} bs={bs}")
        dev, host, maxc, scale = _case(seed, ctx, Hq, Hkv, D, bs)
        assert ops.opscale_attn_decode_workspace_size(len(ctx), Hq, D, maxc) <= 64 << 20
        out = torch.full_like(dev["q"], float("nan"))
        ops.opscale_attn_decode_noalloc(dev["q"], dev["kc"], dev["vc"], dev["table"], dev["ctx"], maxc, scale, out)
        ref_ws = ops.opscale_attn_decode(dev["q"], dev["kc"], dev["vc"], dev["table"], dev["ctx"], maxc, scale)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_ws), name  # same kernels, same partition
        ref = oracle.attn_decode(host["q"], host["kc"], host["vc"], host["table"], host["ctx"], scale)
        assert_close(f64(out.cpu()), ref, "bf16", f"attn_decode_noalloc {name}")


def test_noalloc_decode_rejects_sizes_beyond_its_scratch(ops):
    """B = 2048, Hq = 64, D = 128 needs 4 (256 + 2048) 64 (128 + 2) bytes of
    partials (76.7 MB), more than the 64 MiB the library holds."""
    import torch
    B, Hq, Hkv, D, bs = 2048, 64, 8, 128, 16
    need = ops.opscale_attn_decode_workspace_size(B, Hq, D, 16)
    assert need > ops.opscale_attn_decode_noalloc_max_bytes()
    q = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(B, bs, Hkv, D, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    table = torch.arange(B, dtype=torch.int32, device="cuda").view(B, 1)
    ctxs = torch.full((B,), 16, dtype=torch.int32, device="cuda")
    out = torch.full_like(q, 7.0)
    with pytest.raises(ops.OpscaleError) as ex:
        ops.opscale_attn_decode_noalloc(q, kc, vc, table, ctxs, 16, 1.0 / math.sqrt(D), out)
    assert ex.value.status == ops.OPSCALE_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing was enqueued
