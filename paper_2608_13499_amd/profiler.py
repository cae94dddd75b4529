"""Operator Profiler (Section 4.2): per-operator compute time T_v, memory M_v
and communication payload C_v over the (batch B, sequence length L) space,
built from a sparse random sample instead of an exhaustive sweep.

* Sampling: random points, log-uniform in B and L, inside the profiled domain
  (prefill: B sequences of L tokens each with B * L capped; decode: B
  sequences with a context of L keys), plus the domain's corners so that
  every later query is an interpolation.
* Interpolation: the operators that work token by token (the norms, the
  linears, SiLU-mul, RoPE, the cache write) depend on (B, L) only through
  their token count (B * L in prefill, B in decode), so their T_v is
  interpolated piecewise linearly in log tokens, from samples spread
  log-uniformly over the token range.  Attention depends on B and L apart:
  piecewise linear over the Delaunay triangulation of the sampled points in
  (log B, log L).  Both work on log T_v, so power laws are reproduced
  exactly; a 2-D query outside the sampled hull takes the nearest sample.
* Structural equivalence: a profile is keyed by the operator's structure (its
  kind, phase, the shapes that do not vary with B and L, and dtype), so the 32
  identical layers of an 8B model, or two models sharing an operator shape,
  are profiled once.
* Measurement: every sample is one `opscale_op_profile` call (warmup, then
  iterations timed alone with device events, each after a flush of the
  last-level cache); T_v is the median.  M_v (weight + transient bytes) and
  C_v (bytes handed to the next operator) come from the same call.

Everything that runs on the GPU here is a library entry point; this module
only chooses the points, allocates the operands and fits the interpolant.
"""
from __future__ import annotations

import dataclasses
import json
import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

# ------------------------------------------------------------ signatures ----
PREFILL, DECODE = "prefill", "decode"


@dataclasses.dataclass(frozen=True)
class OpSignature:
    """The structure of one operator: what decides its profile besides (B, L)."""
    kind: str                      # rmsnorm | add_rmsnorm | linear | swiglu | rope | reshape_and_cache |
    #                                attn_prefill | attn_decode
    phase: str                     # prefill | decode
    params: Tuple[Tuple[str, int], ...]
    dtype: str = "bf16"

    def key(self) -> str:
        return f"{self.phase}/{self.kind}/" + ",".join(f"{k}={v}" for k, v in self.params) + f"/{self.dtype}"

    def p(self, name: str) -> int:
        return dict(self.params)[name]


def layer_operators(shape, dtype: str = "bf16", block_size: int = 16) -> List[Tuple[str, OpSignature]]:
    """The operators of one decoder layer (prefill and decode phases), named
    as in a layer's dataflow, with their structural signatures."""
    H, Hq, Hkv, D, F = shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn
    out = []
    for phase in (PREFILL, DECODE):
        def sig(kind, **kw):
            return OpSignature(kind, phase, tuple(sorted(kw.items())), dtype)
        attn = (sig("attn_prefill", Hq=Hq, Hkv=Hkv, D=D) if phase == PREFILL else
                sig("attn_decode", Hq=Hq, Hkv=Hkv, D=D, bs=block_size))
        out += [
            (f"{phase}.input_norm", sig("add_rmsnorm", H=H)),
            (f"{phase}.qkv_proj", sig("linear", N=(Hq + 2 * Hkv) * D, K=H)),
            (f"{phase}.rope", sig("rope", Hq=Hq, Hkv=Hkv, D=D)),
            (f"{phase}.kv_cache_write", sig("reshape_and_cache", Hkv=Hkv, D=D, bs=block_size)),
            (f"{phase}.attention", attn),
            (f"{phase}.o_proj", sig("linear", N=H, K=Hq * D)),
            (f"{phase}.post_attn_norm", sig("add_rmsnorm", H=H)),
            (f"{phase}.gate_up_proj", sig("linear", N=2 * F, K=H)),
            (f"{phase}.act_mul", sig("swiglu", F=F)),
            (f"{phase}.down_proj", sig("linear", N=H, K=F)),
        ]
    return out


# ----------------------------------------------------------------- domain ----
@dataclasses.dataclass(frozen=True)
class Domain:
    """B in [b_min, b_max], L in [l_min, l_max], and B * L <= max_tokens (the
    token budget of one prefill call; decode keeps B * L keys in its cache)."""
    b_min: int
    b_max: int
    l_min: int
    l_max: int
    max_tokens: int

    def contains(self, B: int, L: int) -> bool:
        return (self.b_min <= B <= self.b_max and self.l_min <= L <= self.l_max and B * L <= self.max_tokens)

    def corners(self) -> List[Tuple[int, int]]:
        pts = [(self.b_min, self.l_min), (self.b_max, self.l_min), (self.b_min, self.l_max), (self.b_max, self.l_max)]
        # where the token cap cuts the rectangle, its two cut points
        out = [p for p in pts if self.contains(*p)]
        if not self.contains(self.b_max, self.l_max):
            out.append((max(self.b_min, self.max_tokens // self.l_max), self.l_max))
            out.append((self.b_max, max(self.l_min, self.max_tokens // self.b_max)))
        return sorted(set(out))


def sample_points(domain: Domain, n: int, seed: int, with_corners: bool = True) -> List[Tuple[int, int]]:
    """n distinct points, log-uniform in B and L, inside the domain (plus its
    corners when asked)."""
    rng = np.random.default_rng(seed)
    pts = set(domain.corners()) if with_corners else set()
    target = len(pts) + n
    tries = 0
    while len(pts) < target and tries < 100000:
        tries += 1
        B = int(round(math.exp(rng.uniform(math.log(domain.b_min), math.log(domain.b_max)))))
        L = int(round(math.exp(rng.uniform(math.log(domain.l_min), math.log(domain.l_max)))))
        if domain.contains(B, L):
            pts.add((B, L))
    return sorted(pts)


# ----------------------------------------------------------- interpolant ----
class PiecewiseModel:
    """Piecewise-linear interpolation of log(value) over the Delaunay
    triangulation of the sample points in (log B, log L)."""

    def __init__(self, points: Sequence[Tuple[int, int]], values: Sequence[float]):
        from scipy.interpolate import LinearNDInterpolator, NearestNDInterpolator
        pts = np.log(np.asarray(points, np.float64))
        vals = np.log(np.asarray(values, np.float64))
        if len(pts) < 3:
            raise ValueError("at least 3 sample points are needed")
        self._lin = LinearNDInterpolator(pts, vals)
        self._near = NearestNDInterpolator(pts, vals)
        self.points = [tuple(map(int, p)) for p in points]
        self.values = [float(v) for v in values]

    def predict(self, B, L):
        q = np.log(np.column_stack([np.atleast_1d(B), np.atleast_1d(L)]).astype(np.float64))
        v = self._lin(q)
        miss = ~np.isfinite(v)
        if miss.any():
            v[miss] = self._near(q[miss])
        out = np.exp(v)
        return float(out[0]) if np.ndim(B) == 0 else out


# Operators whose work is a function of the token count alone.
TOKENWISE_KINDS = frozenset({"rmsnorm", "add_rmsnorm", "linear", "swiglu", "rope", "reshape_and_cache"})


def tokens_of(phase: str, B: int, L: int) -> int:
    """Token rows one call processes: B prompts of L tokens in prefill, one new
    token per sequence in decode."""
    return B * L if phase == PREFILL else B


class TokenModel:
    """Piecewise-linear interpolation of log(value) in log(tokens), with the
    end segments extended past the sampled range."""

    def __init__(self, phase: str, points: Sequence[Tuple[int, int]], values: Sequence[float]):
        self.phase = phase
        toks = np.array([tokens_of(phase, B, L) for B, L in points], np.float64)
        logv = np.log(np.asarray(values, np.float64))
        xs = np.unique(np.log(toks))
        if len(xs) < 2:
            raise ValueError("at least 2 distinct token counts are needed")
        # equal token counts (different B, L): their mean log value
        self._x = xs
        self._y = np.array([logv[np.isclose(np.log(toks), x)].mean() for x in xs])
        self.points = [tuple(map(int, p)) for p in points]
        self.values = [float(v) for v in values]

    def predict(self, B, L):
        q = np.log(np.array([tokens_of(self.phase, b, l) for b, l in
                             zip(np.atleast_1d(B), np.atleast_1d(L))], np.float64))
        x, y = self._x, self._y
        v = np.interp(q, x, y)
        lo, hi = q < x[0], q > x[-1]
        v[lo] = y[0] + (q[lo] - x[0]) * (y[1] - y[0]) / (x[1] - x[0])
        v[hi] = y[-1] + (q[hi] - x[-1]) * (y[-1] - y[-2]) / (x[-1] - x[-2])
        out = np.exp(v)
        return float(out[0]) if np.ndim(B) == 0 else out


def sample_points_for(sig: "OpSignature", domain: "Domain", n: int, seed: int,
                      with_corners: bool = True) -> List[Tuple[int, int]]:
    """Sample points of an operator: for a token-wise operator, token counts
    log-uniform over the domain's range (each realized by a (B, L) inside
    it), with the smallest and largest counts; otherwise `sample_points`."""
    if sig.kind not in TOKENWISE_KINDS:
        return sample_points(domain, n, seed, with_corners)
    rng = np.random.default_rng(seed)
    if sig.phase == PREFILL:
        t_lo, t_hi = domain.b_min * domain.l_min, min(domain.max_tokens, domain.b_max * domain.l_max)
    else:
        t_lo, t_hi = domain.b_min, domain.b_max
    pts = set()
    if with_corners:
        pts.add((domain.b_min, domain.l_min))
        pts.add((t_hi // domain.l_min if sig.phase == PREFILL and t_hi // domain.l_min <= domain.b_max else
                 domain.b_max, t_hi // domain.b_max if sig.phase == PREFILL else domain.l_min))
    seen = {tokens_of(sig.phase, *p) for p in pts}
    # stratified: one point in each of n equal slices of the log token range
    # (a random place in it), so no stretch is left bare; a slice too narrow
    # to hold a new integer count is skipped
    for k in range(n):
        for _ in range(50):
            u = (k + rng.uniform()) / n
            T = int(round(math.exp(math.log(t_lo) + u * (math.log(t_hi) - math.log(t_lo)))))
            if sig.phase == PREFILL:
                # a prompt count that can hold T tokens, then the length
                b_hi = min(domain.b_max, T // domain.l_min)
                b_lo = max(domain.b_min, -(-T // domain.l_max))
                if b_lo > b_hi:
                    continue
                B = int(round(math.exp(rng.uniform(math.log(b_lo), math.log(b_hi)))))
                L = max(domain.l_min, min(domain.l_max, int(round(T / B))))
            else:
                B, L = T, int(round(math.exp(rng.uniform(math.log(domain.l_min), math.log(domain.l_max)))))
            if domain.contains(B, L) and tokens_of(sig.phase, B, L) not in seen:
                pts.add((B, L))
                seen.add(tokens_of(sig.phase, B, L))
                break
    return sorted(pts)


def relative_errors(model: PiecewiseModel, points, measured) -> np.ndarray:
    pred = np.asarray([model.predict(B, L) for B, L in points])
    meas = np.asarray(measured, np.float64)
    return np.abs(pred - meas) / meas


# ---------------------------------------------------------------- samples ----
@dataclasses.dataclass
class Sample:
    B: int
    L: int
    us_median: float
    us_p10: float
    us_p90: float
    weight_bytes: int
    transient_bytes: int
    io_bytes: int
    alg_flops: float
    alg_bytes: float


@dataclasses.dataclass
class OpProfile:
    signature: OpSignature
    samples: List[Sample]

    def time_model(self):
        pts, vals = [(s.B, s.L) for s in self.samples], [s.us_median for s in self.samples]
        if self.signature.kind in TOKENWISE_KINDS:
            return TokenModel(self.signature.phase, pts, vals)
        return PiecewiseModel(pts, vals)

    def memory_model(self) -> PiecewiseModel:
        return PiecewiseModel([(s.B, s.L) for s in self.samples],
                              [max(1, s.weight_bytes + s.transient_bytes) for s in self.samples])

    def to_json(self) -> dict:
        sg = self.signature
        return {"kind": sg.kind, "phase": sg.phase, "params": [list(p) for p in sg.params], "dtype": sg.dtype,
                "samples": [dataclasses.asdict(s) for s in self.samples]}

    @staticmethod
    def from_json(d: dict) -> "OpProfile":
        sg = OpSignature(d["kind"], d["phase"], tuple((k, int(v)) for k, v in d["params"]), d["dtype"])
        return OpProfile(sg, [Sample(**s) for s in d["samples"]])


class ProfileStore:
    """Profiles by structural key; operators with equal structure share one."""

    def __init__(self):
        self.profiles: Dict[str, OpProfile] = {}

    def has(self, sig: OpSignature) -> bool:
        return sig.key() in self.profiles

    def get(self, sig: OpSignature) -> OpProfile:
        return self.profiles[sig.key()]

    def put(self, prof: OpProfile):
        self.profiles[prof.signature.key()] = prof

    def profile_layers(self, ops: Iterable[Tuple[str, OpSignature]], measure, points_for) -> Dict[str, str]:
        """Profile every operator of `ops` whose structure is not yet in the
        store; returns name -> structural key (the reuse map)."""
        used = {}
        for name, sig in ops:
            if not self.has(sig):
                pts = points_for(sig)
                self.put(OpProfile(sig, [measure(sig, B, L) for B, L in pts]))
            used[name] = sig.key()
        return used

    def to_json(self) -> str:
        return json.dumps({k: p.to_json() for k, p in self.profiles.items()})

    @staticmethod
    def from_json(text: str) -> "ProfileStore":
        st = ProfileStore()
        for _, d in json.loads(text).items():
            st.put(OpProfile.from_json(d))
        return st


# ------------------------------------------------------------ measurement ----
class Measurer:
    """Builds the operands of one operator at (B, L) on the GPU and runs
    `opscale_op_profile` on them."""

    def __init__(self, warmup: int = 3, iters: int = 10, flush_mib: int = 512, seed: int = 0,
                 rope_theta: float = 500000.0):
        import torch
        from . import _lib as L
        self.L, self.torch = L, torch
        self.warmup, self.iters, self.seed, self.theta = warmup, iters, seed, rope_theta
        self.flush = torch.empty(flush_mib << 20, dtype=torch.uint8, device="cuda") if flush_mib else None
        self._weights = {}

    def _rand(self, shape, std=1.0, mean=0.0):
        torch = self.torch
        g = torch.Generator(device="cuda")
        g.manual_seed(self.seed * 1000003 + int(np.prod(shape)) % 1000003)
        t = torch.empty(*shape, dtype=torch.float32, device="cuda").normal_(mean, std, generator=g)
        return t.to(torch.bfloat16 if self._dt == "bf16" else torch.float32)

    def __call__(self, sig: OpSignature, B: int, L_: int) -> Sample:
        desc, keep = self.build(sig, B, L_)
        p = self.L.opscale_op_profile(desc, self.warmup, self.iters, self.flush)
        if p.us_median < 200.0 and self.iters < 40:
            # short launches vary more from one to the next: take more of them
            p = self.L.opscale_op_profile(desc, 0, 40, self.flush)
        del keep
        return Sample(B, L_, p.us_median, p.us_p10, p.us_p90, int(p.weight_bytes), int(p.transient_bytes),
                      int(p.io_bytes), float(p.alg_flops), float(p.alg_bytes))

    def build(self, sig: OpSignature, B: int, L_: int):
        """The operands of `sig` at (B, L) on the GPU and its descriptor:
        (desc, tensors to keep alive while the descriptor is used)."""
        torch, L = self.torch, self.L
        self._dt = sig.dtype
        T = B * L_ if sig.phase == PREFILL else B
        k = sig.kind
        keep = []
        if k in ("rmsnorm", "add_rmsnorm"):
            H = sig.p("H")
            x, r, w = self._rand((T, H)), self._rand((T, H)), self._rand((H,), 0.02, 1.0)
            y = torch.empty_like(x)
            keep = [x, r, w, y]
            desc = L.desc_add_rmsnorm(x, r, w, y) if k == "add_rmsnorm" else L.desc_rmsnorm(x, w, y)
        elif k == "linear":
            N, K = sig.p("N"), sig.p("K")
            key = (sig.dtype, N, K)
            if key not in self._weights:
                self._weights[key] = self._rand((N, K), 0.02)
            x = self._rand((T, K))
            y = torch.empty(T, N, dtype=x.dtype, device="cuda")
            keep = [x, y]
            desc = L.desc_linear(x, self._weights[key], y)
        elif k == "swiglu":
            F = sig.p("F")
            gu = self._rand((T, 2 * F))
            out = torch.empty(T, F, dtype=gu.dtype, device="cuda")
            keep = [gu, out]
            desc = L.desc_swiglu(gu, out)
        elif k in ("rope", "attn_prefill"):
            Hq, Hkv, D = sig.p("Hq"), sig.p("Hkv"), sig.p("D")
            qkv = self._rand((T, (Hq + 2 * Hkv) * D))
            q = qkv[:, : Hq * D].view(T, Hq, D)
            kk = qkv[:, Hq * D:(Hq + Hkv) * D].view(T, Hkv, D)
            v = qkv[:, (Hq + Hkv) * D:].view(T, Hkv, D)
            if k == "rope":
                pos = torch.arange(T, dtype=torch.int32, device="cuda") % L_ if sig.phase == PREFILL else \
                    torch.full((T,), L_ - 1, dtype=torch.int32, device="cuda")
                keep = [qkv, pos]
                desc = L.desc_rope(q, kk, pos, self.theta)
            else:
                cu = torch.arange(0, T + 1, L_, dtype=torch.int32, device="cuda")
                o = torch.empty(T, Hq, D, dtype=qkv.dtype, device="cuda")
                keep = [qkv, cu, o]
                desc = L.desc_attn_prefill(q, kk, v, o, cu, L_, 1.0 / math.sqrt(D))
        elif k == "reshape_and_cache":
            Hkv, D, bs = sig.p("Hkv"), sig.p("D"), sig.p("bs")
            kv = self._rand((T, 2 * Hkv * D))
            kk = kv[:, : Hkv * D].view(T, Hkv, D)
            v = kv[:, Hkv * D:].view(T, Hkv, D)
            # prefill: B sequences of L tokens; decode: one token per sequence
            # at position L - 1; the cache holds B sequences of L tokens
            nb = B * ((L_ + bs - 1) // bs)
            kc = torch.empty(nb, bs, Hkv, D, dtype=kv.dtype, device="cuda")
            vc = torch.empty_like(kc)
            rng = np.random.default_rng(self.seed)
            perm = rng.permutation(nb * bs)
            slots = perm[:T] if sig.phase == PREFILL else perm[:B]
            sl = torch.from_numpy(slots.astype(np.int32)).cuda()
            keep = [kv, kc, vc, sl]
            desc = L.desc_reshape_and_cache(kk, v, kc, vc, sl)
        elif k == "attn_decode":
            Hq, Hkv, D, bs = sig.p("Hq"), sig.p("Hkv"), sig.p("D"), sig.p("bs")
            nblk = (L_ + bs - 1) // bs
            nb = B * nblk
            kc = self._rand((nb, bs, Hkv, D))
            vc = self._rand((nb, bs, Hkv, D))
            rng = np.random.default_rng(self.seed)
            table = torch.from_numpy(rng.permutation(nb).astype(np.int32).reshape(B, nblk)).cuda()
            ctx = torch.full((B,), L_, dtype=torch.int32, device="cuda")
            q = self._rand((B, Hq, D))
            o = torch.empty_like(q)
            ws = torch.empty(L.opscale_attn_decode_workspace_size(B, Hq, D, L_), dtype=torch.uint8, device="cuda")
            keep = [kc, vc, table, ctx, q, o, ws]
            desc = L.desc_attn_decode(q, kc, vc, table, ctx, o, L_, 1.0 / math.sqrt(D), ws)
        else:
            raise ValueError(f"unknown operator kind {k}")
        return desc, keep


def domain_for(sig: OpSignature, max_prefill_tokens: int = 65536) -> Domain:
    if sig.phase == PREFILL:
        return Domain(1, 64, 16, 8192, max_prefill_tokens)
    return Domain(1, 256, 16, 8192, 256 * 8192)


def evaluate(prof: OpProfile, heldout: List[Sample]) -> dict:
    err = relative_errors(prof.time_model(), [(s.B, s.L) for s in heldout], [s.us_median for s in heldout])
    return {"n_samples": len(prof.samples), "n_heldout": len(heldout), "mean_rel_err": float(err.mean()),
            "p90_rel_err": float(np.quantile(err, 0.9)), "max_rel_err": float(err.max())}


def main(argv: Optional[Sequence[str]] = None) -> int:
    import argparse
    import sys
    from .layer import LayerShape
    ap = argparse.ArgumentParser(description="Profile the operators of one decoder layer and report the "
                                             "prediction error of the sparse profiles on held-out points.")
    ap.add_argument("--hidden", type=int, default=4096)
    ap.add_argument("--heads", type=int, default=32)
    ap.add_argument("--kv-heads", type=int, default=8)
    ap.add_argument("--head-dim", type=int, default=128)
    ap.add_argument("--ffn", type=int, default=14336)
    ap.add_argument("--samples", type=int, default=20, help="random samples per token-wise operator (plus the "
                                                             "ends of its token range)")
    ap.add_argument("--samples-2d", type=int, default=96, help="random samples per attention operator (plus the "
                                                               "domain corners)")
    ap.add_argument("--heldout", type=int, default=12)
    ap.add_argument("--max-prefill-tokens", type=int, default=65536)
    ap.add_argument("--layers", type=int, default=32, help="layers of the model (they share profiles)")
    ap.add_argument("--only", default="", help="comma-separated operator names to profile (default: all)")
    ap.add_argument("--out", default="", help="write the profile store as JSON here")
    a = ap.parse_args(argv)
    shape = LayerShape(a.hidden, a.heads, a.kv_heads, a.head_dim, a.ffn)
    meas = Measurer()
    store = ProfileStore()
    ops = [(f"layer{i}.{n}", s) for i in range(a.layers) for n, s in layer_operators(shape)]
    if a.only:
        keep = set(a.only.split(","))
        ops = [(n, s) for n, s in ops if n.split(".", 1)[1] in keep]
    uniq = {}
    for n, s in ops:
        uniq.setdefault(s.key(), (n, s))
    print(f"{len(ops)} operator instances, {len(uniq)} distinct structures to profile", file=sys.stderr, flush=True)
    results = {}
    pooled = []
    for key, (name, sig) in uniq.items():
        dom = domain_for(sig, a.max_prefill_tokens)
        pts = sample_points_for(sig, dom, a.samples if sig.kind in TOKENWISE_KINDS else a.samples_2d, seed=1)
        ho_pts = [p for p in sample_points(dom, a.heldout, seed=2, with_corners=False) if p not in set(pts)]
        prof = OpProfile(sig, [meas(sig, B, L) for B, L in pts])
        store.put(prof)
        ho = [meas(sig, B, L) for B, L in ho_pts]
        results[key] = evaluate(prof, ho)
        pooled += list(relative_errors(prof.time_model(), [(h.B, h.L) for h in ho], [h.us_median for h in ho]))
        r = results[key]
        print(f"{name.split('.', 1)[1]:28s} {sig.key():70s} samples {r['n_samples']:3d} held-out {r['n_heldout']:3d} "
              f"mean err {100 * r['mean_rel_err']:5.1f}%  p90 {100 * r['p90_rel_err']:5.1f}%", flush=True)
    used = store.profile_layers(ops, meas, lambda s: [])  # every structure is in the store: nothing re-measured
    pooled = np.asarray(pooled)
    print(json.dumps({"instances": len(ops), "profiled_structures": len(store.profiles),
                      "reused_instances": len(used) - len(store.profiles),
                      "heldout_predictions": int(pooled.size), "mean_rel_err": float(pooled.mean()),
                      "p90_rel_err": float(np.quantile(pooled, 0.9))}), flush=True)
    if a.out:
        with open(a.out, "w") as f:
            f.write(store.to_json())
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
