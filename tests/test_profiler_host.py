"""Host-side checks of the operator profiler (no GPU): the interpolant, the
sampling domain, structural-equivalence reuse and serialization."""
import math

import numpy as np
import pytest

from paper_2608_13499_amd import profiler as pr
from paper_2608_13499_amd.layer import LayerShape

SHAPE_8B = LayerShape(4096, 32, 8, 128, 14336)


def test_power_laws_are_reproduced_exactly():
    # T = c * B^a * L^b is linear in (log B, log L): the interpolant is exact inside the hull
    dom = pr.Domain(1, 64, 16, 8192, 65536)
    pts = pr.sample_points(dom, 12, seed=3)
    f = lambda B, L: 3.5 * B ** 0.9 * L ** 1.7
    m = pr.PiecewiseModel(pts, [f(B, L) for B, L in pts])
    for B, L in pr.sample_points(dom, 30, seed=4, with_corners=False):
        assert abs(m.predict(B, L) / f(B, L) - 1) < 1e-9


def test_interpolant_passes_through_samples_and_stays_finite_outside():
    pts = [(1, 16), (64, 16), (1, 8192), (8, 8192), (64, 1024), (7, 300)]
    vals = [5.0, 40.0, 900.0, 3000.0, 2000.0, 77.0]
    m = pr.PiecewiseModel(pts, vals)
    for (B, L), v in zip(pts, vals):
        assert abs(m.predict(B, L) - v) / v < 1e-12
    assert np.isfinite(m.predict(200, 10))  # outside: nearest sample


def test_piecewise_error_shrinks_with_more_samples():
    dom = pr.Domain(1, 64, 16, 8192, 65536)
    f = lambda B, L: B * L * (1 + 0.3 * math.sin(math.log(B * L)))  # not a power law
    ho = pr.sample_points(dom, 200, seed=9, with_corners=False)
    errs = []
    for n in (6, 24, 96):
        pts = pr.sample_points(dom, n, seed=5)
        m = pr.PiecewiseModel(pts, [f(*p) for p in pts])
        errs.append(float(np.mean(pr.relative_errors(m, ho, [f(*p) for p in ho]))))
    assert errs[2] < errs[0]


def test_domain_and_sampling():
    dom = pr.Domain(1, 64, 16, 8192, 65536)
    c = dom.corners()
    assert (1, 16) in c and (64, 16) in c and (1, 8192) in c
    assert (8, 8192) in c and (64, 1024) in c        # where B * L = 65536 cuts the rectangle
    assert all(dom.contains(*p) for p in c)
    pts = pr.sample_points(dom, 20, seed=1)
    assert len(pts) == 20 + len(c) and all(dom.contains(*p) for p in pts)
    assert pts == pr.sample_points(dom, 20, seed=1)   # reproducible
    assert pts != pr.sample_points(dom, 20, seed=2)


def test_layer_structures_and_reuse():
    ops = pr.layer_operators(SHAPE_8B)
    assert len(ops) == 20                             # 10 operators per phase
    keys = {s.key() for _, s in ops}
    # the two norms of a phase share a structure; the four linears do not
    assert len(keys) == 18
    names = dict(ops)
    assert names["prefill.input_norm"] == names["prefill.post_attn_norm"]
    assert names["prefill.o_proj"] != names["prefill.down_proj"]
    assert names["prefill.qkv_proj"].p("N") == (32 + 16) * 128
    # 32 identical layers: every structure is measured once
    calls = []

    def fake_measure(sig, B, L):
        calls.append((sig.key(), B, L))
        return pr.Sample(B, L, float(B * L), 0, 0, 0, 0, 0, 0, 0)

    store = pr.ProfileStore()
    model_ops = [(f"layer{i}.{n}", s) for i in range(32) for n, s in ops]
    used = store.profile_layers(model_ops, fake_measure, lambda s: [(1, 16), (4, 64), (2, 1000)])
    assert len(used) == 640 and len(store.profiles) == 18
    assert len(calls) == 18 * 3
    # a second model with the same operator shapes reuses all of them
    store.profile_layers([(f"other.{n}", s) for n, s in ops], fake_measure, lambda s: [(1, 16)])
    assert len(calls) == 18 * 3
    # a model whose attention groups differ re-profiles only the operators that changed
    ops_mha = pr.layer_operators(LayerShape(4096, 32, 32, 128, 14336))
    store.profile_layers(ops_mha, fake_measure, lambda s: [(1, 16), (4, 64), (2, 1000)])
    changed = {s.key() for _, s in ops_mha} - {s.key() for _, s in ops}
    assert len(calls) == 18 * 3 + 3 * len(changed)
    assert all(k.split("/")[1] in ("linear", "rope", "reshape_and_cache", "attn_prefill", "attn_decode")
               for k in changed)


def test_store_json_roundtrip():
    sig = pr.OpSignature("linear", "prefill", (("K", 4096), ("N", 6144)), "bf16")
    prof = pr.OpProfile(sig, [pr.Sample(1, 16, 10.0, 9.0, 11.0, 100, 200, 50, 1e9, 1e6),
                              pr.Sample(8, 128, 30.0, 29.0, 31.0, 100, 900, 400, 8e9, 2e6),
                              pr.Sample(2, 4096, 80.0, 79.0, 81.0, 100, 3000, 1200, 3e10, 9e6)])
    st = pr.ProfileStore()
    st.put(prof)
    st2 = pr.ProfileStore.from_json(st.to_json())
    p2 = st2.get(sig)
    assert p2.signature == sig and p2.samples == prof.samples
    assert abs(p2.time_model().predict(8, 128) - 30.0) < 1e-9


def test_token_model_for_tokenwise_operators():
    """Norms, linears, SiLU-mul, RoPE and the cache write are interpolated in
    their token count: exact on a power law of the tokens, through every
    sample, and equal at equal token counts whatever (B, L) holds them."""
    ops = dict(pr.layer_operators(SHAPE_8B))
    for name in ("prefill.qkv_proj", "prefill.input_norm", "decode.down_proj", "decode.kv_cache_write"):
        sig = ops[name]
        dom = pr.domain_for(sig)
        pts = pr.sample_points_for(sig, dom, 20, seed=1)
        tok = lambda B, L: pr.tokens_of(sig.phase, B, L)
        f = lambda B, L: 2.0 * tok(B, L) ** 0.8
        prof = pr.OpProfile(sig, [pr.Sample(B, L, f(B, L), 0, 0, 0, 0, 0, 0, 0) for B, L in pts])
        m = prof.time_model()
        assert isinstance(m, pr.TokenModel)
        for B, L in pts:
            assert abs(m.predict(B, L) / f(B, L) - 1) < 1e-9
        for B, L in pr.sample_points(dom, 40, seed=7, with_corners=False):
            assert abs(m.predict(B, L) / f(B, L) - 1) < 1e-9
        if sig.phase == pr.PREFILL:
            assert abs(m.predict(4, 1024) - m.predict(64, 64)) < 1e-9 * m.predict(64, 64)
        else:
            assert m.predict(17, 100) == m.predict(17, 8000)  # decode: one token per sequence
    # attention keeps the 2-D model
    assert isinstance(pr.OpProfile(ops["prefill.attention"], [pr.Sample(B, L, float(B * L * L), 0, 0, 0, 0, 0, 0, 0)
                      for B, L in [(1, 16), (64, 16), (1, 8192), (8, 8192)]]).time_model(), pr.PiecewiseModel)


def test_tokenwise_sampling_covers_the_token_range():
    """One sample in each of n equal slices of the log token range, plus the
    two ends; every point inside the domain and distinct in tokens."""
    ops = dict(pr.layer_operators(SHAPE_8B))
    for name, n in (("prefill.gate_up_proj", 20), ("decode.o_proj", 20), ("prefill.act_mul", 8)):
        sig = ops[name]
        dom = pr.domain_for(sig)
        pts = pr.sample_points_for(sig, dom, n, seed=3)
        toks = sorted(pr.tokens_of(sig.phase, B, L) for B, L in pts)
        assert all(dom.contains(B, L) for B, L in pts) and len(set(toks)) == len(toks)
        lo, hi = toks[0], toks[-1]
        assert lo == (dom.b_min * dom.l_min if sig.phase == pr.PREFILL else dom.b_min)
        assert hi == (dom.max_tokens if sig.phase == pr.PREFILL else dom.b_max)
        # gap between neighbours in log tokens: at most two slices, plus the
        # rounding of a count to an integer (half a token at each end)
        slice_ = (math.log(hi) - math.log(lo)) / n
        for a, b in zip(toks, toks[1:]):
            assert math.log(b / a) <= 2 * slice_ + math.log((a + 0.5) / a) + math.log(b / (b - 0.5)) + 1e-9
        assert pts == pr.sample_points_for(sig, dom, n, seed=3)
