"""Spatial sharing on the GPU: CU-masked streams really confine kernels to
their share (the placement probe reads each workgroup's XCD and CU), the
co-run profile agrees with the oracle's summary of its own raw launch times,
and latency responds to the share as the paper describes (a compute-bound
prefill operator slows down in proportion, a 1-token decode operator hardly).
"""
import numpy as np
import pytest

from oracle import spatial as osp
from parity_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as P
    P.load()
    return P


@pytest.fixture(scope="module")
def layout(ops):
    n, x, il = ops.opscale_cu_layout()
    say(f"CU layout: {n} CUs, {x} XCDs, mask {'interleaved' if il else 'blocked'} over the XCDs")
    return n, x, il


def _cu_keys(ops, stream, nwg=4096, spins=2):
    """The (XCD, CU) of every workgroup of one probe launch on `stream`."""
    import torch
    out = torch.zeros(nwg, 2, dtype=torch.int32, device="cuda")
    ops.opscale_cu_probe(out, spins, stream=stream)
    torch.cuda.synchronize()
    a = out.cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    return {(int(x), int((h >> 8) & 0xFF)) for x, h in a}


def test_layout(layout):
    n, x, il = layout
    assert n == 256 and x == 8 and il in (0, 1)


def test_stream_keeps_its_mask(ops, layout):
    n, x, il = layout
    mask = ops.opscale_cu_mask_build(n, x, il, 0, 64)
    s = ops.opscale_cu_stream_create(mask)
    try:
        assert ops.opscale_cu_stream_mask(s, len(mask)) == mask
    finally:
        ops.opscale_cu_stream_destroy(s)


def test_probe_sees_every_cu(ops, layout):
    import torch
    keys = _cu_keys(ops, torch.cuda.current_stream().cuda_stream, nwg=8192)
    say(f"probe on the default stream: {len(keys)} distinct CUs")
    assert len(keys) == layout[0]
    assert sorted({x for x, _ in keys}) == list(range(layout[1]))


@pytest.mark.parametrize("k", [13, 64, 128])
def test_shares_are_disjoint_and_balanced(ops, layout, k):
    n, x, il = layout
    sa = ops.opscale_cu_stream_create(ops.opscale_cu_mask_build(n, x, il, 0, k))
    sb = ops.opscale_cu_stream_create(ops.opscale_cu_mask_build(n, x, il, k, n - k))
    try:
        ka, kb = _cu_keys(ops, sa), _cu_keys(ops, sb)
    finally:
        ops.opscale_cu_stream_destroy(sa)
        ops.opscale_cu_stream_destroy(sb)
    per = np.bincount([xx for xx, _ in ka], minlength=x)
    say(f"share of {k} CUs: probe used {len(ka)} CUs (per XCD {per.tolist()}); complement {len(kb)}")
    assert len(ka) == k and len(kb) == n - k
    assert not ka & kb
    assert per.max() - per.min() <= 1


def _norm_and_linear(ops):
    import torch
    g = torch.Generator(device="cuda").manual_seed(7)
    x = torch.randn(8192, 4096, device="cuda", generator=g).to(torch.bfloat16)
    w = torch.ones(4096, device="cuda", dtype=torch.bfloat16)
    y = torch.empty_like(x)
    a = torch.randn(1024, 4096, device="cuda", generator=g).to(torch.bfloat16)
    W = (0.02 * torch.randn(4096, 4096, device="cuda", generator=g)).to(torch.bfloat16)
    c = torch.empty(1024, 4096, device="cuda", dtype=torch.bfloat16)
    keep = (x, w, y, a, W, c)
    return ops.desc_rmsnorm(x, w, y), ops.desc_linear(a, W, c), keep


def test_corun_matches_oracle_summary(ops, layout):
    n, x, il = layout
    da, db, keep = _norm_and_linear(ops)
    sa = ops.opscale_cu_stream_create(ops.opscale_cu_mask_build(n, x, il, 0, n // 2))
    sb = ops.opscale_cu_stream_create(ops.opscale_cu_mask_build(n, x, il, n // 2, n - n // 2))
    try:
        r, tr = ops.opscale_corun_profile(da, sa, db, sb, warmup=3, iso_iters=12, window_ms=5.0,
                                          max_launches=1024, trace=True)
    finally:
        ops.opscale_cu_stream_destroy(sa)
        ops.opscale_cu_stream_destroy(sb)
    ref = osp.corun_summary(tr["a_start"], tr["a_end"], tr["b_start"], tr["b_end"], tr["a_iso"], tr["b_iso"])
    say(f"co-run rmsnorm | linear on 128 | 128 CUs: launches {r.n_a} / {r.n_b}, overlapped {r.overlap_a} / "
        f"{r.overlap_b}, T {r.a_iso_us:.1f} / {r.b_iso_us:.1f} us, T~ {r.a_co_us:.1f} / {r.b_co_us:.1f} us, "
        f"I {r.interference_a:.3f} / {r.interference_b:.3f}")
    assert (r.overlap_a, r.overlap_b) == (ref["overlap_a"], ref["overlap_b"])
    for f in ("a_iso_us", "b_iso_us", "a_co_us", "b_co_us", "interference_a", "interference_b"):
        assert getattr(r, f) == pytest.approx(ref[f], rel=1e-6), f
    assert r.overlap_a >= 4 and r.overlap_b >= 4
    assert 0.8 < r.interference_a < 5 and 0.8 < r.interference_b < 5
    # the launches of each stream are back to back and in order
    for s, e in ((tr["a_start"], tr["a_end"]), (tr["b_start"], tr["b_end"])):
        s, e = np.asarray(s), np.asarray(e)
        assert np.all(e > s) and np.all(s[1:] == e[:-1])


def test_corun_needs_two_streams(ops, layout):
    da, db, keep = _norm_and_linear(ops)
    import torch
    s = torch.cuda.current_stream().cuda_stream
    with pytest.raises(ops.OpscaleError):
        ops.opscale_corun_profile(da, s, db, s)


def test_share_sensitivity_prefill_vs_decode(ops, layout):
    """Section 2.1's contrast: a 2K-token projection slows down markedly on a
    smaller share (a quarter of the CUs: about x2.4, less than x4 because at
    2048 rows the GEMM's 192 tiles do not fill all 256 CUs), a 1-token one,
    bound by streaming the weights, much less."""
    import torch
    n, x, il = layout
    W = (0.02 * torch.randn(6144, 4096, device="cuda")).to(torch.bfloat16)
    res = {}
    for tokens in (2048, 1):
        a = torch.randn(tokens, 4096, device="cuda").to(torch.bfloat16)
        c = torch.empty(tokens, 6144, device="cuda", dtype=torch.bfloat16)
        d = ops.desc_linear(a, W, c)
        t = {}
        for k in (n // 4, n):
            s = ops.opscale_cu_stream_create(ops.opscale_cu_mask_build(n, x, il, 0, k))
            try:
                t[k] = ops.opscale_op_profile(d, warmup=3, iters=15, stream=s).us_median
            finally:
                ops.opscale_cu_stream_destroy(s)
        res[tokens] = t[n // 4] / t[n]
        say(f"QKV linear, {tokens} tokens: {t[n]:.1f} us on all CUs, {t[n // 4]:.1f} us on a quarter "
            f"(x{res[tokens]:.2f})")
    assert res[2048] > 2.0
    assert res[1] < res[2048]
