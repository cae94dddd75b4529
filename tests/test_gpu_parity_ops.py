"""GPU parity of every operator against the fp64 oracle, at sizes the oracle
evaluates in full: the tiny fp32 decoder layer (tolerance 1e-5) and bf16 shapes
that span several kernel tiles with ragged tails in every dimension
(tolerance 2e-2), plus the degenerate cases (single row, single key, empty
prompts, zero-length contexts, invalid page ids).  All calls go through the C
ABI via the ctypes binding."""
import math

import numpy as np
import pytest

import oracle
import workloads as wl
from parity_util import assert_close, cuda, f64, gen, say, torch_dtype

pytestmark = pytest.mark.gpu


TILES = {"256x256": 0, "192x256": 1, "256x128": 2, "256x256w8": 3}  # opscale_tune GEMM_TILE values
SCHEDULES = {"grid": 0, "list": 1}                   # opscale_tune PREFILL_SCHEDULE values


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as ops
    ops.load()
    return ops


# ------------------------------------------------------------------ RMSNorm --
@pytest.mark.parametrize("dtype,M,H", [
    ("f32", 128, 256), ("f32", 5, 4), ("bf16", 37, 4096), ("bf16", 3, 8192),
    ("bf16", 9, 24), ("bf16", 2, 24576), ("bf16", 1, 4096), ("f32", 7, 16384 + 4),
])
def test_rmsnorm(ops, dtype, M, H):
    import torch
    say(f"rmsnorm {dtype} M={M} H={H}")
    x = gen(11, "x", (M, H), dtype)
    w = gen(11, "w_norm", (H,), dtype, std=0.02, mean=1.0)
    y = ops.opscale_rmsnorm(cuda(x), cuda(w), eps=1e-5)
    torch.cuda.synchronize()
    assert_close(f64(y.cpu()), oracle.rmsnorm(f64(x), f64(w), 1e-5), dtype, "rmsnorm")


def test_rmsnorm_inplace_and_unit_gain(ops):
    import torch
    x = gen(12, "x", (64, 4096), "bf16")
    xd = cuda(x)
    ops.opscale_rmsnorm(xd, cuda(torch.ones(4096, dtype=torch.bfloat16)), y=xd, eps=0.0)
    torch.cuda.synchronize()
    y = f64(xd.cpu())
    # unit gain, eps 0: every row has RMS 1 up to bf16 output rounding
    rms = np.sqrt(np.mean(y * y, axis=1))
    assert np.abs(rms - 1).max() < 4e-3
    assert_close(y, oracle.rmsnorm(f64(x), np.ones(4096), 0.0), "bf16", "in-place rmsnorm")


# ------------------------------------------------------------------- linear --
@pytest.mark.parametrize("dtype,M,N,K,bias", [
    ("f32", 128, 768, 256, False), ("f32", 128, 256, 256, False), ("f32", 128, 1376, 256, False),
    ("f32", 128, 256, 688, False), ("f32", 3, 12, 20, True),
    ("bf16", 300, 264, 200, False), ("bf16", 513, 1024, 4096, False), ("bf16", 1, 256, 64, False),
    ("bf16", 257, 520, 136, True), ("bf16", 64, 6144, 4096, False), ("bf16", 40, 256, 14336, False),
    ("bf16", 1000, 768, 8, False),
])
def test_linear(ops, dtype, M, N, K, bias):
    import torch
    say(f"linear {dtype} M={M} N={N} K={K} bias={bias}")
    x = gen(21, "x", (M, K), dtype)
    W = gen(21, "w_qkv", (N, K), dtype, std=0.02)
    b = gen(21, "bias", (N,), dtype) if bias else None
    y = ops.opscale_linear(cuda(x), cuda(W), None if b is None else cuda(b))
    torch.cuda.synchronize()
    assert_close(f64(y.cpu()), oracle.linear(f64(x), f64(W), None if b is None else f64(b)), dtype, "linear")


@pytest.mark.parametrize("tile", ["256x256", "192x256", "256x128", "256x256w8"])
@pytest.mark.parametrize("M,N,K,bias", [(300, 264, 200, True), (513, 1024, 4096, False), (1, 256, 64, False),
                                        (700, 520, 136, False)])
def test_linear_each_tile(ops, tune, tile, M, N, K, bias):
    """Every bf16 tile shape the dispatcher can pick, with ragged M, N and K."""
    import torch
    say(f"linear bf16 tile={tile} M={M} N={N} K={K} bias={bias}")
    tune(gemm_tile=TILES[tile])
    x = gen(23, "x", (M, K), "bf16")
    W = gen(23, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(23, "bias", (N,), "bf16") if bias else None
    y = ops.opscale_linear(cuda(x), cuda(W), None if b is None else cuda(b))
    torch.cuda.synchronize()
    assert_close(f64(y.cpu()), oracle.linear(f64(x), f64(W), None if b is None else f64(b)), "bf16", "linear")


@pytest.mark.parametrize("M,N,K,bias", [
    (1, 256, 64, False), (3, 40, 96, True), (16, 6144, 4096, False), (17, 520, 128, True), (33, 8, 32, False),
    (64, 4096, 14336, False), (100, 1000, 4096, True), (129, 264, 256, False), (256, 6144, 4096, False),
    (256, 4104, 32, True),
])
@pytest.mark.parametrize("ng", [1, 2])
def test_linear_small_m(ops, tune, ng, M, N, K, bias):
    """The decode-batch path (M <= 256, K % 32 == 0), forced on, with 16 and
    32 columns per workgroup: every row-group count, N tails shorter than one
    column group, K of one k-step per wave and fewer k-steps than waves."""
    import torch
    tune(gemm_skinny=1, skinny_ng=ng)
    say(f"linear bf16 small-M NG={ng} M={M} N={N} K={K} bias={bias}")
    x = gen(24, "x", (M, K), "bf16")
    W = gen(24, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(24, "bias", (N,), "bf16") if bias else None
    y = ops.opscale_linear(cuda(x), cuda(W), None if b is None else cuda(b))
    y2 = ops.opscale_linear(cuda(x), cuda(W), None if b is None else cuda(b))
    torch.cuda.synchronize()
    assert torch.equal(y, y2)  # fixed reduction order
    assert_close(f64(y.cpu()), oracle.linear(f64(x), f64(W), None if b is None else f64(b)), "bf16", "linear")


@pytest.mark.parametrize("M,N,K,bias", [
    (256, 6144, 4096, False), (100, 520, 1032, True), (17, 4096, 14336, False), (200, 1000, 2048, True),
    (64, 8, 1024, False), (700, 4096, 4096, True), (64, 6144, 4096, True), (65, 1000, 2048, False),
    (96, 4096, 4096, False), (128, 28672, 1024, True), (256, 4096, 14336, False),
    (200, 16648, 1024, True), (256, 28672, 4096, False),
])
def test_linear_split_k(ops, tune, M, N, K, bias):
    """Decode-sized M with K split over workgroups (fp32 partials summed in
    split order), on each tile the path picks (64 or 128 rows up to 256, 256
    rows with 256 or 128 columns above): ragged M, N and K, a K range that
    does not divide evenly, bias; 129-256 rows whose 128-row tiles fill the
    GPU without a split (the last two cases); bitwise equal across calls.
    The partials live in the caller's workspace (poisoned before the call:
    its contents on entry must not matter); without one the same shapes take
    an unsplit path."""
    import torch
    tune(gemm_skinny=0, gemm_decode=0)
    say(f"linear bf16 split-K M={M} N={N} K={K} bias={bias}")
    x = gen(25, "x", (M, K), "bf16")
    W = gen(25, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(25, "bias", (N,), "bf16") if bias else None
    args = (cuda(x), cuda(W), None if b is None else cuda(b))
    need = ops.opscale_linear_workspace_size(M, N, K)
    ws = torch.full((max(need, 16),), 0x7f, dtype=torch.uint8, device="cuda")  # fp32 3.4e38 if read
    y = ops.opscale_linear(*args, workspace=ws)
    y2 = ops.opscale_linear(*args, workspace=ws)
    y0 = ops.opscale_linear(*args, workspace=False)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    ref = oracle.linear(f64(x), f64(W), None if b is None else f64(b))
    assert_close(f64(y.cpu()), ref, "bf16", "linear")
    assert_close(f64(y0.cpu()), ref, "bf16", "linear without a workspace")


@pytest.mark.parametrize("M,N,K,bias", [
    (256, 6144, 4096, False), (256, 4096, 4096, True), (256, 4096, 14336, False), (256, 28672, 4096, False),
    (200, 1000, 2048, True), (129, 264, 256, False), (100, 520, 1088, True), (65, 136, 64, True),
    (33, 8, 512, False), (1, 256, 64, False), (64, 6144, 4096, True), (256, 4104, 576, True),
    (256, 256, 16384, False), (128, 1304, 832, False),
])
def test_linear_decode_batch(ops, tune, M, N, K, bias):
    """The decode-batch kernel (weights streamed into registers, 128 columns
    and all M rows per workgroup), forced on: every row-block count (M up to
    64, 128, 256 and ragged between), N tails down to 8 columns and waves
    with no weight rows, K of one slice, ranges that are not a multiple of the
    8-slice round and uneven K ranges, K split over workgroups through the
    caller's workspace (poisoned: its contents on entry must not matter) or
    not at all; bitwise equal across calls.  Without a workspace a shape that
    would split takes another path."""
    import torch
    tune(gemm_decode=1)
    say(f"linear bf16 decode-batch M={M} N={N} K={K} bias={bias}")
    x = gen(28, "x", (M, K), "bf16")
    W = gen(28, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(28, "bias", (N,), "bf16") if bias else None
    args = (cuda(x), cuda(W), None if b is None else cuda(b))
    need = ops.opscale_linear_workspace_size(M, N, K)
    ws = torch.full((max(need, 16),), 0x7f, dtype=torch.uint8, device="cuda")
    y = ops.opscale_linear(*args, workspace=ws)
    y2 = ops.opscale_linear(*args, workspace=ws)
    y0 = ops.opscale_linear(*args, workspace=False)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    ref = oracle.linear(f64(x), f64(W), None if b is None else f64(b))
    assert_close(f64(y.cpu()), ref, "bf16", "linear")
    assert_close(f64(y0.cpu()), ref, "bf16", "linear without a workspace")


@pytest.mark.parametrize("M,N,K,bias", [(777, 1304, 2120, True), (2048, 6144, 4096, False), (256, 512, 64, True),
                                        (1300, 1000, 2056, True), (520, 384, 8256, False)])
def test_linear_four_and_eight_waves_agree(ops, tune, M, N, K, bias):
    """The 256x256 tile as four waves of 128x128 (accumulators in AGPRs) and
    as eight waves of 128x64 accumulate every output over the same k-steps
    with the same MFMA, so their results are bitwise equal; both match the
    oracle.  The four-wave ring gives the two-slice lead to x on the first,
    third and fifth shapes (tile groups of at most four tile-rows) and to W
    on the second and fourth (groups of more rows); the ragged K of the first
    and fourth ends in a partial slice, the fifth runs 129 slices and the
    third a single one."""
    import torch
    say(f"linear bf16 four vs eight waves M={M} N={N} K={K} bias={bias}")
    x = gen(27, "x", (M, K), "bf16")
    W = gen(27, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(27, "bias", (N,), "bf16") if bias else None
    args = (cuda(x), cuda(W), None if b is None else cuda(b))
    tune(gemm_tile=TILES["256x256"])
    y4 = ops.opscale_linear(*args)
    tune(gemm_tile=TILES["256x256w8"])
    y8 = ops.opscale_linear(*args)
    torch.cuda.synchronize()
    assert torch.equal(y4.view(torch.int16), y8.view(torch.int16))
    assert_close(f64(y4.cpu()), oracle.linear(f64(x), f64(W), None if b is None else f64(b)), "bf16", "linear")


@pytest.mark.parametrize("tile,M,N,K,bias", [("256x256", 4352, 4096, 1024, True), ("256x256", 4300, 4104, 2056, False),
                                             ("192x256", 4352, 4096, 1024, False),
                                             ("256x256w8", 4300, 4104, 2056, True)])
def test_linear_split_tail(ops, tune, tile, M, N, K, bias):
    """More tiles than CUs with the last round at most half full: those tiles
    run as 2-4 K ranges (fp32 partials summed in split order) in the same
    launch as the others.  Ragged M, N and K, bias; bitwise equal across
    calls; the same result with the split tail turned off and with no
    workspace (which also plans no split)."""
    import torch
    say(f"linear bf16 split tail tile={tile} M={M} N={N} K={K} bias={bias}")
    tune(gemm_tile=TILES[tile])
    assert ops.opscale_linear_workspace_size(M, N, K) > 0
    x = gen(26, "x", (M, K), "bf16")
    W = gen(26, "w_qkv", (N, K), "bf16", std=0.02)
    b = gen(26, "bias", (N,), "bf16") if bias else None
    args = (cuda(x), cuda(W), None if b is None else cuda(b))
    y = ops.opscale_linear(*args)
    y2 = ops.opscale_linear(*args)
    yn = ops.opscale_linear(*args, workspace=False)
    tune(gemm_tail=0)
    y0 = ops.opscale_linear(*args)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    ref = oracle.linear(f64(x), f64(W), None if b is None else f64(b))
    assert_close(f64(y.cpu()), ref, "bf16", "linear split tail")
    assert_close(f64(y0.cpu()), ref, "bf16", "linear without split tail")
    assert torch.equal(y0, yn)  # both unsplit


def test_linear_identity_weight(ops):
    """W = I (bf16-exact) returns x exactly: no accumulation rounding occurs."""
    import torch
    x = gen(22, "x", (300, 512), "bf16")
    W = torch.eye(512, dtype=torch.bfloat16)
    y = ops.opscale_linear(cuda(x), cuda(W))
    torch.cuda.synchronize()
    assert torch.equal(y.cpu(), x)


# ------------------------------------------------------------------- SwiGLU --
@pytest.mark.parametrize("dtype,M,F", [("f32", 128, 688), ("bf16", 33, 1000), ("bf16", 1, 14336),
                                       ("bf16", 700, 8), ("f32", 3, 4)])
def test_swiglu(ops, dtype, M, F):
    import torch
    say(f"swiglu {dtype} M={M} F={F}")
    u = gen(31, "gate_up", (M, 2 * F), dtype, std=3.0)
    out = ops.opscale_swiglu(cuda(u))
    torch.cuda.synchronize()
    assert_close(f64(out.cpu()), oracle.swiglu(f64(u)), dtype, "swiglu")


# -------------------------------------------------------- prefill attention --
def _prefill_case(ops, dtype, lens, Hq, Hkv, D, causal, packed, seed=41):
    import torch
    lens = np.asarray(lens, np.int64)
    cu = wl.cu_seqlens(lens)
    T = int(cu[-1])
    if packed:  # views into one [T, (Hq + 2 Hkv) D] tensor, as after the QKV linear
        qkv = gen(seed, "q", (T, (Hq + 2 * Hkv) * D), dtype)
        qd = cuda(qkv)
        q = qd[:, : Hq * D].view(T, Hq, D)
        k = qd[:, Hq * D:(Hq + Hkv) * D].view(T, Hkv, D)
        v = qd[:, (Hq + Hkv) * D:].view(T, Hkv, D)
        qh = f64(qkv[:, : Hq * D]).reshape(T, Hq, D)
        kh = f64(qkv[:, Hq * D:(Hq + Hkv) * D]).reshape(T, Hkv, D)
        vh = f64(qkv[:, (Hq + Hkv) * D:]).reshape(T, Hkv, D)
    else:
        qc, kc, vc = (gen(seed, "q", (T, Hq, D), dtype), gen(seed, "k", (T, Hkv, D), dtype),
                      gen(seed, "v", (T, Hkv, D), dtype))
        q, k, v = cuda(qc), cuda(kc), cuda(vc)
        qh, kh, vh = f64(qc), f64(kc), f64(vc)
    scale = 1.0 / math.sqrt(D)
    out = ops.opscale_attn_prefill(q, k, v, cuda(torch.from_numpy(cu)), int(max(1, lens.max())), scale,
                                   causal)
    torch.cuda.synchronize()
    ref = oracle.attn_prefill(qh, kh, vh, cu, scale, causal)
    return f64(out.cpu()), ref


@pytest.mark.parametrize("dtype,lens,Hq,Hkv,D,causal,packed", [
    ("f32", [128], 4, 4, 64, True, False),
    ("f32", [5, 70, 0, 1], 4, 2, 128, True, True),
    ("f32", [33, 7], 2, 1, 64, False, False),
    ("bf16", [1, 17, 64, 65, 130, 0, 300], 8, 2, 128, True, False),
    ("bf16", [128, 40, 1], 4, 4, 64, True, False),
    ("bf16", [200, 31, 97], 16, 2, 128, True, True),
    ("bf16", [77, 3, 150], 6, 2, 128, True, False),
    ("bf16", [100, 1, 64], 8, 2, 128, False, False),
    ("bf16", [513], 2, 2, 64, True, True),
])
def test_attn_prefill(ops, dtype, lens, Hq, Hkv, D, causal, packed):
    say(f"attn_prefill {dtype} lens={lens} Hq={Hq} Hkv={Hkv} D={D} causal={causal} packed={packed}")
    got, ref = _prefill_case(ops, dtype, lens, Hq, Hkv, D, causal, packed)
    assert_close(got, ref, dtype, "attn_prefill")


@pytest.mark.parametrize("lens,Hq,Hkv,D", [
    ([1, 17, 64, 65, 130, 0, 300, 33], 8, 2, 128),   # ragged, G = 4 (32-query tiles)
    ([96, 96, 96], 4, 2, 64),                        # uniform, G = 2 (64-query tiles)
    ([900, 5, 1, 260], 3, 3, 128),                   # G = 1 (128-query tiles)
    ([1, 2, 3, 17] * 20 + [700], 8, 1, 64),          # 81 prompts: more than one wave of 64
    # a long prompt before a short one, two equal prompts, one tile and a key:
    # the K/V loads in these tiles must land where their stage says (a missing
    # wait state before a load once wrote some of them to the previous load's
    # place, in the grid schedule only)
    ([300, 1], 4, 1, 128),
    ([130, 130], 4, 1, 128),
    ([65], 4, 1, 128),
])
def test_attn_prefill_schedules(ops, tune, lens, Hq, Hkv, D):
    """Both schedules (grid; level-major work list) against the oracle, and
    bitwise equal to each other (each tile is computed the same way)."""
    outs = {}
    for sched in ("grid", "list"):
        tune(prefill_schedule=SCHEDULES[sched])
        say(f"attn_prefill bf16 schedule={sched} lens={lens} Hq={Hq} Hkv={Hkv} D={D}")
        got, ref = _prefill_case(ops, "bf16", lens, Hq, Hkv, D, True, True)
        assert_close(got, ref, "bf16", f"attn_prefill ({sched})")
        outs[sched] = got
    assert np.array_equal(outs["grid"], outs["list"])


def test_attn_prefill_many_prompts(ops, tune):
    """More prompts than the work list holds in LDS: the launcher takes the grid
    even when the list is asked for."""
    tune(prefill_schedule=SCHEDULES["list"])
    say("attn_prefill bf16 1101 prompts")
    lens = ([1, 2, 3, 17] * 276)[:1101]
    got, ref = _prefill_case(ops, "bf16", lens, 8, 2, 128, True, True)
    assert_close(got, ref, "bf16", "attn_prefill 1101 prompts")


def test_attn_prefill_1024_prompts_list(ops, tune):
    """The largest batch the work list takes (1024 prompts, 16 waves of 64)."""
    tune(prefill_schedule=SCHEDULES["list"])
    say("attn_prefill bf16 1024 prompts (work list)")
    lens = ([1, 40, 3, 97, 0, 64] * 171)[:1024]
    got, ref = _prefill_case(ops, "bf16", lens, 8, 2, 64, True, True)
    assert_close(got, ref, "bf16", "attn_prefill 1024 prompts")


def test_attn_prefill_single_key_returns_v(ops):
    """Prompts of length 1: softmax over one key is exactly 1, output == v."""
    import torch
    lens = [1] * 9
    cu = wl.cu_seqlens(lens)
    q = gen(42, "q", (9, 8, 128), "bf16")
    k = gen(42, "k", (9, 2, 128), "bf16")
    v = gen(42, "v", (9, 2, 128), "bf16")
    out = ops.opscale_attn_prefill(cuda(q), cuda(k), cuda(v), cuda(torch.from_numpy(cu)), 1, 0.088)
    torch.cuda.synchronize()
    exp = v.repeat_interleave(4, dim=1)
    assert torch.equal(out.cpu(), exp)


# --------------------------------------------------------- decode attention --
def _decode_case(ops, dtype, ctx, Hq, Hkv, D, bs, seed=51, bad_block=False, max_context_len=None):
    import torch
    ctx = np.asarray(ctx, np.int64)
    rng = wl.rng_for(seed, "block_table")
    table, nb = wl.paged_cache_layout(ctx, bs, rng, extra_blocks=3)
    if bad_block:
        table = table.copy()
        table[0, 0] = nb + 5  # out of range: the keys of this page are skipped
    kc = gen(seed, "k_cache", (nb, bs, Hkv, D), dtype)
    vc = gen(seed, "v_cache", (nb, bs, Hkv, D), dtype)
    q = gen(seed, "q", (len(ctx), Hq, D), dtype)
    scale = 1.0 / math.sqrt(D)
    maxc = int(max(1, ctx.max())) if max_context_len is None else max_context_len
    out = ops.opscale_attn_decode(cuda(q), cuda(kc), cuda(vc), cuda(torch.from_numpy(table)),
                                  cuda(torch.from_numpy(ctx.astype(np.int32))), maxc, scale)
    torch.cuda.synchronize()
    kh, vh = f64(kc), f64(vc)
    if bad_block:
        # expected: the same sequence without the keys of its first page
        ref = oracle.attn_decode(f64(q), kh, vh, np.concatenate([table[:, 1:], table[:, :1]], 1),
                                 np.concatenate([[ctx[0] - bs], ctx[1:]]), scale)
        ref[1:] = oracle.attn_decode(f64(q)[1:], kh, vh, table[1:], ctx[1:], scale)
    else:
        ref = oracle.attn_decode(f64(q), kh, vh, table, ctx, scale)
    return f64(out.cpu()), ref


@pytest.mark.parametrize("dtype,ctx,Hq,Hkv,D,bs", [
    ("f32", [1, 16, 17, 600, 0], 8, 2, 128, 16),
    ("f32", [37, 5], 4, 4, 64, 8),
    ("bf16", [1, 16, 17, 600, 0], 8, 2, 128, 16),
    ("bf16", [1030, 2, 513, 9], 32, 8, 128, 16),
    ("bf16", [40, 300], 4, 4, 64, 16),
    ("bf16", [129, 2049, 31], 16, 2, 128, 32),
    ("bf16", [100, 7], 4, 2, 128, 1),
    ("bf16", [4000, 64], 16, 8, 64, 256),
])
def test_attn_decode(ops, dtype, ctx, Hq, Hkv, D, bs):
    say(f"attn_decode {dtype} ctx={ctx} Hq={Hq} Hkv={Hkv} D={D} bs={bs}")
    got, ref = _decode_case(ops, dtype, ctx, Hq, Hkv, D, bs)
    assert_close(got, ref, dtype, "attn_decode")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attn_decode_invalid_block_is_skipped(ops, dtype):
    say(f"attn_decode invalid block id {dtype}")
    got, ref = _decode_case(ops, dtype, [40, 20], 8, 2, 128, 16, bad_block=True)
    assert_close(got, ref, dtype, "attn_decode bad block")


@pytest.mark.parametrize("name,ctx,maxc", [
    # far fewer 32-key tiles than workgroups: most workgroups have no keys
    ("sparse", [0, 5, 0, 33, 1, 0, 64, 2], 4096),
    ("one long, many short", [9000] + [3] * 39, None),
    # about 1.5 tiles a workgroup: ranges straddle sequence boundaries
    ("straddling", list(np.random.default_rng(8).integers(1, 2000, 100)), None),
    # one workgroup a sequence, each over several 512-key page windows
    ("few workgroups", [3000, 1, 1500, 0, 2047], 1),
    ("all empty", [0, 0, 0], 64),
    # above 512 sequences the plan comes from its own kernel
    ("large batch", list(np.random.default_rng(9).integers(0, 300, 700)), None),
    ("large batch, sparse", [0] * 600 + [40] + [0] * 100 + [1], 2048),
])
def test_attn_decode_balanced_ranges(ops, name, ctx, maxc):
    """Every workgroup takes an equal range of the batch's 32-key tiles; the
    ranges and the merge must cover each sequence's keys exactly once."""
    say(f"attn_decode balanced ranges: {name} (B={len(ctx)})")
    got, ref = _decode_case(ops, "bf16", ctx, 8, 2, 128, 16, seed=len(ctx), max_context_len=maxc)
    assert_close(got, ref, "bf16", f"attn_decode {name}")
    if max(ctx) == 0:
        assert np.all(got == 0)


@pytest.mark.parametrize("bs", [16, 1])
def test_attn_decode_context_beyond_launch_bound(ops, bs):
    """max_context_len only sizes the launch: a longer context is processed in
    several key windows by one split and the result is unchanged."""
    say(f"attn_decode context beyond max_context_len, bs={bs}")
    got, ref = _decode_case(ops, "bf16", [2000, 700, 3], 8, 2, 128, bs, max_context_len=100)
    assert_close(got, ref, "bf16", "attn_decode long context")
