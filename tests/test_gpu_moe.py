"""The mixture-of-experts path on the GPU against the oracle: top-k routing
(ids exact, the decision taken on the same fp32 logits; weights to fp32
rounding) and the fused expert MLPs (bf16 tolerance), on ragged problems
(experts without tokens, one expert with every token, invalid ids, duplicate
routes, one token), at Mixtral-8x7B widths on sampled tokens, and bitwise
repeatability."""
import numpy as np
import pytest

from oracle import moe as om
from parity_util import assert_close, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_13499_amd as P
    P.load()
    return P


def _t(a, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).cuda()


@pytest.mark.parametrize("T,E,k,ren,ties", [(300, 64, 8, True, False), (300, 64, 8, False, True),
                                             (129, 8, 2, True, True), (5, 3, 1, False, False),
                                             (70, 1000, 16, True, False)])
def test_topk_routing(ops, T, E, k, ren, ties):
    import torch
    say(f"moe_topk T={T} E={E} k={k} renormalize={ren} ties={ties}")
    rng = np.random.default_rng(T + E + k)
    lg = rng.normal(size=(T, E)).astype(np.float32)
    if ties:
        lg = np.round(lg * 2) / 2  # many equal logits
    ids, w = ops.opscale_moe_topk(_t(lg, torch.float32), k, ren)
    torch.cuda.synchronize()
    rid, rw = om.topk_route(lg, k, ren)
    assert np.array_equal(ids.cpu().numpy(), rid)
    assert np.allclose(w.cpu().numpy(), rw, rtol=2e-6, atol=1e-7)


def _moe_case(ops, T, H, F, E, k, seed, ids=None, wts=None):
    import torch
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(T, H)).astype(np.float32)
    w1 = (rng.normal(size=(E, 2 * F, H)) / np.sqrt(H)).astype(np.float32)
    w2 = (rng.normal(size=(E, H, F)) / np.sqrt(F)).astype(np.float32)
    if ids is None:
        ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]) if k <= E else rng.integers(0, E, (T, k))
    if wts is None:
        wts = rng.uniform(0.1, 1.0, size=(T, k)).astype(np.float32)
    xb, w1b, w2b = (_t(a, torch.bfloat16) for a in (x, w1, w2))
    out = ops.opscale_fused_moe(xb, w1b, w2b, _t(np.asarray(ids, np.int32), torch.int32),
                                _t(np.asarray(wts, np.float32), torch.float32))
    out2 = ops.opscale_fused_moe(xb, w1b, w2b, _t(np.asarray(ids, np.int32), torch.int32),
                                 _t(np.asarray(wts, np.float32), torch.float32))
    torch.cuda.synchronize()
    assert torch.equal(out, out2)  # ordered sort and sums: bitwise repeatable
    f64 = lambda t_: t_.float().cpu().numpy().astype(np.float64)
    ref = om.fused_moe(f64(xb), f64(w1b), f64(w2b), ids, np.asarray(wts, np.float32))
    return f64(out), ref


@pytest.mark.parametrize("fuse", [-1, 0])
@pytest.mark.parametrize("T,H,F,E,k", [(37, 64, 96, 8, 2), (300, 128, 256, 64, 8), (1, 64, 64, 4, 1),
                                        (600, 256, 512, 3, 2), (257, 96, 40, 16, 4)])
def test_fused_moe(ops, tune, fuse, T, H, F, E, k):
    """Both paths: the SwiGLU fused into the gate-up GEMM's epilogue (gate
    and up rows interleaved), and the separate gate-up output plus SwiGLU."""
    tune(moe_fuse=fuse)  # -1: automatic (fused at these sizes); 0: unfused
    say(f"fused_moe T={T} H={H} F={F} E={E} topk={k} fuse={fuse}")
    got, ref = _moe_case(ops, T, H, F, E, k, seed=T * 7 + E)
    assert_close(got, ref, "bf16", "fused_moe")


def test_fused_moe_one_hot_expert(ops):
    """Every token to expert 2 (600 rows: three 256-row tiles), the others empty."""
    say("fused_moe all tokens to one expert")
    T = 600
    got, ref = _moe_case(ops, T, 128, 128, 6, 1, seed=5, ids=np.full((T, 1), 2))
    assert_close(got, ref, "bf16", "fused_moe one expert")


def test_fused_moe_invalid_and_duplicate_routes(ops):
    """Ids outside [0, E) contribute nothing; two slots may name one expert."""
    say("fused_moe invalid and duplicate ids")
    T, E = 50, 5
    rng = np.random.default_rng(9)
    ids = rng.integers(0, E, size=(T, 3))
    ids[::7, 0] = -1
    ids[3::11, 2] = E + 3
    ids[::5, 1] = ids[::5, 0]
    got, ref = _moe_case(ops, T, 64, 64, E, 3, seed=9, ids=ids)
    assert_close(got, ref, "bf16", "fused_moe invalid ids")
    dead = np.all((ids < 0) | (ids >= E), axis=1)
    assert np.all(got[dead] == 0)


def test_fused_moe_mixtral_width_sampled(ops):
    """Mixtral-8x7B expert widths (H 4096, F 14336), two experts, top-2, 256
    tokens; the oracle on 6 sampled tokens (rows are independent)."""
    import torch
    say("fused_moe Mixtral widths, 256 tokens, sampled rows")
    T, H, F, E, k = 256, 4096, 14336, 2, 2
    g = torch.Generator(device="cuda").manual_seed(3)
    x = torch.randn(T, H, device="cuda", generator=g).to(torch.bfloat16)
    w1 = (torch.randn(E, 2 * F, H, device="cuda", generator=g) / 64).to(torch.bfloat16)
    w2 = (torch.randn(E, H, F, device="cuda", generator=g) / 120).to(torch.bfloat16)
    rng = np.random.default_rng(3)
    ids = np.stack([rng.permutation(E) for _ in range(T)]).astype(np.int32)
    wts = rng.uniform(0.2, 1.0, (T, k)).astype(np.float32)
    out = ops.opscale_fused_moe(x, w1, w2, _t(ids, torch.int32), _t(wts, torch.float32))
    torch.cuda.synchronize()
    rows = [0, 1, 77, 128, 200, 255]
    f64 = lambda t_: t_.float().cpu().numpy().astype(np.float64)
    ref = om.fused_moe(f64(x[rows]), f64(w1), f64(w2), ids[rows], wts[rows])
    assert_close(f64(out[rows]), ref, "bf16", "fused_moe Mixtral rows")


def test_fused_moe_rejects(ops):
    import torch
    x = torch.zeros(4, 64, dtype=torch.float32, device="cuda")
    w1 = torch.zeros(2, 128, 64, dtype=torch.float32, device="cuda")
    w2 = torch.zeros(2, 64, 64, dtype=torch.float32, device="cuda")
    ids = torch.zeros(4, 1, dtype=torch.int32, device="cuda")
    wts = torch.ones(4, 1, dtype=torch.float32, device="cuda")
    with pytest.raises(ops.OpscaleError):
        ops.opscale_fused_moe(x, w1, w2, ids, wts)  # fp32: bf16 only
