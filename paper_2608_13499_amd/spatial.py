"""Spatial sharing of one GPU between operators.

The paper runs colocated operators on separate streams that each own a share
of the SMs.  It characterizes how each operator's latency depends on its share
(Section 2.1, "Sensitivity to SM Core Allocation": a 2K-token prefill against
a 1-token decode).  Its placement models colocation with an interference
factor per operator pair (Section 4.4, Eq. 5).  The factor is
I_{d,v}(b, p) = T~_v(b, p) / T_v(b, p): v's latency while its partner runs,
over v's latency alone at the same share p.  It is swept at 5 % share
granularity and stored in a lookup table that snaps a query to the nearest
profiled grid point.  A three-way colocation is the product of the pairwise
factors, and the model is validated on held-out measurements (Section 5.7,
Table 2: 5 % mean and 9.4 % P90 slowdown-prediction error).

The MI355X counterpart of an SM share is a stream with a CU mask
(`opscale_cu_stream_create`).  A share of k CUs takes k positions of the
balanced order, which spreads it evenly over the 8 XCDs (`opscale_cu_mask_build`
with the mask layout measured by `opscale_cu_layout`).  Two colocated
operators get the complementary position ranges [0, k) and [k, 256).  Every
measurement is a library call (`opscale_op_profile` on a masked stream, or
`opscale_corun_profile` on two).  This module chooses the points, allocates
the operands (through the profiler's `Measurer`) and keeps the table.
"""
from __future__ import annotations

import dataclasses
import json
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .profiler import DECODE, PREFILL, OpSignature

SHARE_STEP = 0.05
SHARE_GRID = tuple(round(SHARE_STEP * i, 2) for i in range(1, 20))  # 5 % ... 95 %


# ------------------------------------------------------------ CU shares ----
@dataclasses.dataclass(frozen=True)
class CULayout:
    num_cus: int
    num_xcds: int
    interleaved: int

    def mask(self, first: int, count: int) -> List[int]:
        from . import _lib as L
        return L.opscale_cu_mask_build(self.num_cus, self.num_xcds, self.interleaved, first, count)

    def split(self, p: float) -> int:
        """CUs of the first of two complementary shares at fraction p (both >= 1)."""
        return int(min(self.num_cus - 1, max(1, round(p * self.num_cus))))


def cu_layout() -> CULayout:
    from . import _lib as L
    return CULayout(*L.opscale_cu_layout())


class CUStream:
    """A stream masked to positions [first, first + count) of the balanced order."""

    def __init__(self, layout: CULayout, first: int, count: int):
        from . import _lib as L
        self._L = L
        self.first, self.count = first, count
        self.handle = L.opscale_cu_stream_create(layout.mask(first, count))

    def close(self):
        if self.handle:
            self._L.opscale_cu_stream_destroy(self.handle)
            self.handle = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


# ------------------------------------------------------------ workloads ----
@dataclasses.dataclass(frozen=True)
class Workload:
    """An operator of the layer at one load b: prefill kinds take b tokens (one
    prompt of length b), decode kinds b sequences with a fixed context."""
    kind: str
    sig: OpSignature
    context: int = 2048

    def shape(self, b: int) -> Tuple[int, int]:
        return (1, b) if self.sig.phase == PREFILL else (b, self.context)


def llama8b_workloads(dtype: str = "bf16") -> Dict[str, Workload]:
    """The operator kinds of the interference study (Llama-3-8B layer shapes)."""
    def sig(kind, phase, **kw):
        return OpSignature(kind, phase, tuple(sorted(kw.items())), dtype)
    return {
        "norm": Workload("norm", sig("add_rmsnorm", PREFILL, H=4096)),
        "qkv": Workload("qkv", sig("linear", PREFILL, N=6144, K=4096)),
        "attn_prefill": Workload("attn_prefill", sig("attn_prefill", PREFILL, Hq=32, Hkv=8, D=128)),
        "act": Workload("act", sig("swiglu", PREFILL, F=14336)),
        "attn_decode": Workload("attn_decode", sig("attn_decode", DECODE, Hq=32, Hkv=8, D=128, bs=16)),
    }


LOAD_GRID = {"norm": (512, 2048, 8192), "qkv": (128, 512, 2048), "attn_prefill": (256, 1024, 4096),
             "act": (512, 2048, 8192), "attn_decode": (16, 64, 256)}


# --------------------------------------------------------- lookup table ----
def snap(grid: Sequence[float], x: float, log: bool = False):
    """The grid point nearest x (in log space if `log`); ties go to the lower point."""
    pts = sorted(grid)
    dist = [abs(math.log(g) - math.log(x)) if log else abs(g - x) for g in pts]
    best = min(dist)
    return pts[next(i for i, d in enumerate(dist) if d <= best + 1e-12)]


def bracket(grid: Sequence[float], x: float, log: bool = False) -> List[Tuple[float, float]]:
    """The grid points around x with their linear weights (in log space if
    `log`); a single point with weight 1 outside the grid's range."""
    g = sorted(grid)
    f = math.log if log else (lambda z: z)
    if x <= g[0]:
        return [(g[0], 1.0)]
    if x >= g[-1]:
        return [(g[-1], 1.0)]
    for lo, hi in zip(g, g[1:]):
        if lo <= x <= hi:
            w = (f(x) - f(lo)) / (f(hi) - f(lo))
            return [(lo, 1.0 - w), (hi, w)]
    raise ValueError(x)


class InterferenceTable:
    """I_v on the grid (kind_v, b_v, partner kind, partner b, share of v)."""

    def __init__(self, loads: Dict[str, Sequence[int]], shares: Sequence[float] = SHARE_GRID):
        self.loads = {k: tuple(v) for k, v in loads.items()}
        self.shares = tuple(shares)
        self.entries: Dict[Tuple[str, int, str, int, float], float] = {}

    @staticmethod
    def _key(v, bv, u, bu, p):
        return (v, int(bv), u, int(bu), round(float(p), 4))

    def put(self, v: str, bv: int, u: str, bu: int, p: float, factor: float):
        self.entries[self._key(v, bv, u, bu, p)] = float(factor)

    def lookup(self, v: str, bv: float, u: str, bu: float, p: float) -> float:
        """The factor at the nearest profiled grid point (loads in log space);
        if that share was not measured for this pair and loads, the nearest
        share that was."""
        gv, gu = snap(self.loads[v], bv, log=True), snap(self.loads[u], bu, log=True)
        key = self._key(v, gv, u, gu, snap(self.shares, p))
        if key in self.entries:
            return self.entries[key]
        have = [s_ for s_ in self.shares if self._key(v, gv, u, gu, s_) in self.entries]
        if not have:
            raise KeyError(f"no interference factor for {v} (b={gv}) next to {u} (b={gu})")
        return self.entries[self._key(v, gv, u, gu, snap(have, p))]

    def interpolate(self, v: str, bv: float, u: str, bu: float, p: float) -> float:
        """Multilinear interpolation over the grid cell around (log b_v, log b_u,
        p) (clamped to the grid's range), instead of the nearest point."""
        f = 0.0
        for gv, wv in bracket(self.loads[v], bv, log=True):
            for gu, wu in bracket(self.loads[u], bu, log=True):
                for gp, wp in bracket(self.shares, p):
                    if wv * wu * wp:
                        f += wv * wu * wp * self.lookup(v, gv, u, gu, gp)
        return f

    def predict(self, v: str, bv: float, p: float, partners: Sequence[Tuple[str, float]],
                interpolate: bool = False) -> float:
        """Slowdown of v at share p next to one or more partners: the product of
        the pairwise factors (one factor for a pair).  The factors come from the
        nearest grid point, or from interpolation with `interpolate`."""
        get = self.interpolate if interpolate else self.lookup
        f = 1.0
        for u, bu in partners:
            f *= get(v, bv, u, bu, p)
        return f

    def to_json(self) -> str:
        return json.dumps({"loads": self.loads, "shares": self.shares,
                           "entries": [[*k, val] for k, val in sorted(self.entries.items())]})

    @staticmethod
    def from_json(text: str) -> "InterferenceTable":
        d = json.loads(text)
        t = InterferenceTable(d["loads"], d["shares"])
        for v, bv, u, bu, p, val in d["entries"]:
            t.put(v, bv, u, bu, p, val)
        return t


def relative_errors(pred: Sequence[float], meas: Sequence[float]) -> np.ndarray:
    pred, meas = np.asarray(pred, np.float64), np.asarray(meas, np.float64)
    return np.abs(pred - meas) / meas


# ---------------------------------------------------------- measurements ----
class SpatialProfiler:
    """Runs the sensitivity sweep, the pairwise co-runs and the held-out checks."""

    def __init__(self, warmup: int = 3, iters: int = 10, window_ms: float = 8.0, seed: int = 0):
        from .profiler import Measurer
        from . import _lib as L
        self.L = L
        self.meas = Measurer(warmup=warmup, iters=iters, flush_mib=0, seed=seed)
        self.layout = cu_layout()
        self.warmup, self.iters, self.window_ms = warmup, iters, window_ms
        self._ops = {}

    def op(self, w: Workload, b: int):
        key = (w.kind, int(b))
        if key not in self._ops:
            B, Lq = w.shape(int(b))
            self._ops[key] = self.meas.build(w.sig, B, Lq)
        return self._ops[key][0]

    def release(self):
        self._ops.clear()

    def sensitivity(self, ops: Sequence[Tuple[str, Workload, int]], shares: Sequence[float]) -> Dict[str, List]:
        """Latency of each operator on a share of p x 256 CUs (alone), for every p."""
        out = {name: [] for name, _, _ in ops}
        for p in shares:
            k = max(1, round(p * self.layout.num_cus))
            with CUStream(self.layout, 0, k) as s:
                for name, w, b in ops:
                    prof = self.L.opscale_op_profile(self.op(w, b), self.warmup, self.iters, None, stream=s.handle)
                    out[name].append({"share": p, "cus": k, "us": prof.us_median,
                                      "roofline_frac": prof.roofline_frac})
        return out

    def corun(self, wv: Workload, bv: int, wu: Workload, bu: int, p: float, streams=None):
        """One co-run of v on share p and u on the complementary share."""
        k = self.layout.split(p)
        own = streams is None
        if own:
            streams = (CUStream(self.layout, 0, k), CUStream(self.layout, k, self.layout.num_cus - k))
        try:
            r = self.L.opscale_corun_profile(self.op(wv, bv), streams[0].handle, self.op(wu, bu), streams[1].handle,
                                             warmup=self.warmup, iso_iters=self.iters, window_ms=self.window_ms,
                                             max_launches=8192)
        finally:
            if own:
                for s in streams:
                    s.close()
        return r

    def build_table(self, works: Dict[str, Workload], loads: Dict[str, Sequence[int]],
                    shares: Sequence[float] = SHARE_GRID, log=None) -> InterferenceTable:
        """Every unordered kind pair, every load pair, every share (one co-run
        gives the factor of both operators: v at p and u at 1 - p)."""
        table = InterferenceTable(loads, shares)
        kinds = sorted(works)
        pairs = [(a, b) for i, a in enumerate(kinds) for b in kinds[i:]]
        for p in shares:
            k = self.layout.split(p)
            with CUStream(self.layout, 0, k) as sa, CUStream(self.layout, k, self.layout.num_cus - k) as sb:
                for v, u in pairs:
                    for bv in loads[v]:
                        for bu in loads[u]:
                            r = self.corun(works[v], bv, works[u], bu, p, streams=(sa, sb))
                            if r.overlap_a and r.overlap_b:
                                table.put(v, bv, u, bu, p, r.interference_a)
                                table.put(u, bu, v, bv, round(1.0 - p, 4), r.interference_b)
            if log:
                log(f"share {p:.2f}: {len(table.entries)} entries")
        return table

    def validate(self, table: InterferenceTable, works: Dict[str, Workload], n: int, seed: int = 1,
                 log=None) -> dict:
        """Held-out co-runs: random kind pairs at loads between the grid points
        and shares off the 5 % grid; predicted vs measured slowdown."""
        rng = np.random.default_rng(seed)
        kinds = sorted(works)
        rows = []
        for i in range(n):
            v, u = rng.choice(kinds), rng.choice(kinds)
            bv = _offgrid_load(rng, table.loads[v])
            bu = _offgrid_load(rng, table.loads[u])
            p = round(float(rng.integers(2, 38)) * 0.025, 4)  # 5 % ... 92.5 %, half of them off the grid
            r = self.corun(works[v], bv, works[u], bu, p)
            for kind, b in ((v, bv), (u, bu)):  # off-grid operands are not kept
                if b not in table.loads[kind]:
                    self._ops.pop((kind, int(b)), None)
            if not (r.overlap_a and r.overlap_b):
                continue
            q = round(1.0 - self.layout.split(p) / self.layout.num_cus, 4)
            rows.append({"v": v, "bv": bv, "u": u, "bu": bu, "p": p, "q": q,
                         "measured_v": r.interference_a, "predicted_v": table.predict(v, bv, p, [(u, bu)]),
                         "interpolated_v": table.predict(v, bv, p, [(u, bu)], interpolate=True),
                         "measured_u": r.interference_b, "predicted_u": table.predict(u, bu, q, [(v, bv)]),
                         "interpolated_u": table.predict(u, bu, q, [(v, bv)], interpolate=True)})
            if log and (i + 1) % 10 == 0:
                log(f"validated {i + 1}/{n}")
        meas = [r["measured_v"] for r in rows] + [r["measured_u"] for r in rows]
        out = {"rows": rows}
        for tag, col in (("", "predicted"), ("interp_", "interpolated")):
            err = relative_errors([r[col + "_v"] for r in rows] + [r[col + "_u"] for r in rows], meas)
            out.update({"n": len(err), tag + "mean_rel_err": float(err.mean()),
                        tag + "p90_rel_err": float(np.quantile(err, 0.9)), tag + "max_rel_err": float(err.max())})
        return out


def _offgrid_load(rng, grid: Sequence[int]) -> int:
    """A load log-uniform over the grid's range, rounded to a multiple of 16."""
    lo, hi = math.log(min(grid)), math.log(max(grid))
    return int(max(16, round(math.exp(rng.uniform(lo, hi)) / 16) * 16))


# ---------------------------------------------------------------- report ----
def report(result: dict, command: str = "") -> str:
    """A plain-text summary of a `spatial all` result."""
    lines = []
    lay = result.get("layout", {})
    if command:
        lines += ["command:", f"  {command}", ""]
    lines.append(f"layout: {lay.get('num_cus')} CUs, {lay.get('num_xcds')} XCDs, mask "
                 f"{'interleaved' if lay.get('interleaved') else 'blocked'} over the XCDs")
    sens = result.get("sensitivity")
    if sens:
        shares = [r["share"] for r in next(iter(sens.values()))]
        show = [i for i, p in enumerate(shares) if round(p * 100) % 10 == 0 or i == 0]
        lines += ["", "latency on a share of the CUs / latency on all CUs (prefill: one 2048-token prompt; "
                  "decode: one sequence, 2048-token context)",
                  f"{'operator':26s}" + "".join(f"{round(100 * shares[i]):>6d}%" for i in show) + "   all CUs"]
        for name, rows in sens.items():
            base = rows[-1]["us"]
            lines.append(f"{name:26s}" + "".join(f"{rows[i]['us'] / base:7.2f}" for i in show) +
                         f"  {base:7.1f} us")
    tab = result.get("table")
    if tab:
        vals = np.array([e[5] for e in tab["entries"]])
        lines += ["", f"interference table: {len(vals)} factors I = T~/T over kinds {sorted(tab['loads'])}, "
                  f"loads {tab['loads']}, shares 5 % ... 95 %",
                  f"  I: min {vals.min():.3f}  median {np.median(vals):.3f}  p90 {np.quantile(vals, 0.9):.3f}  "
                  f"max {vals.max():.3f}"]
        by_kind = {}
        for v, bv, u, bu, p, val in tab["entries"]:
            by_kind.setdefault((v, u), []).append(val)
        kinds = sorted(tab["loads"])
        lines.append("  median I of the row operator next to the column operator (all loads and shares):")
        lines.append("  " + " " * 14 + "".join(f"{k:>14s}" for k in kinds))
        for v in kinds:
            lines.append(f"  {v:14s}" + "".join(f"{np.median(by_kind.get((v, u), [float('nan')])):14.3f}"
                                                 for u in kinds))
    val = result.get("validation")
    if val:
        lines += ["", f"held-out co-runs (loads between the grid points, shares on and off the 5 % grid): "
                  f"{val['n']} predictions", f"  slowdown prediction error, nearest grid point: mean "
                  f"{100 * val['mean_rel_err']:.1f} %, p90 {100 * val['p90_rel_err']:.1f} %, max "
                  f"{100 * val['max_rel_err']:.1f} %"]
        if "interp_mean_rel_err" in val:
            lines.append(f"  slowdown prediction error, interpolated: mean {100 * val['interp_mean_rel_err']:.1f} %, "
                         f"p90 {100 * val['interp_p90_rel_err']:.1f} %, max {100 * val['interp_max_rel_err']:.1f} %")
    return "\n".join(lines) + "\n"


# ------------------------------------------------------------------- CLI ----
def main(argv: Optional[Sequence[str]] = None) -> int:
    import argparse
    import sys
    import time
    ap = argparse.ArgumentParser(description="CU-share sensitivity and pairwise interference (Eq. 5)")
    ap.add_argument("what", choices=["sensitivity", "table", "all", "report"])
    ap.add_argument("--input", help="report: the JSON a previous run wrote")
    ap.add_argument("--out", default="spatial.json")
    ap.add_argument("--heldout", type=int, default=60)
    ap.add_argument("--window-ms", type=float, default=8.0)
    args = ap.parse_args(argv)
    if args.what == "report":
        with open(args.input) as f:
            sys.stdout.write(report(json.load(f), "python -m paper_2608_13499_amd.spatial all --out <json>"))
        return 0
    t0 = time.time()

    def log(msg):
        print(f"[{time.time() - t0:7.1f}s] {msg}", flush=True)

    sp = SpatialProfiler(window_ms=args.window_ms)
    log(f"layout {sp.layout}")
    result = {"layout": dataclasses.asdict(sp.layout)}
    works = llama8b_workloads()
    if args.what in ("sensitivity", "all"):
        from .layer import LayerShape
        from .profiler import layer_operators
        shape = LayerShape(4096, 32, 8, 128, 14336)
        ops = []
        for name, sig in layer_operators(shape):
            wl = Workload(name, sig)
            ops.append((name, wl, 2048 if sig.phase == PREFILL else 1))
        shares = [round(0.05 * i, 2) for i in range(1, 21)]
        result["sensitivity"] = sp.sensitivity(ops, shares)
        sp.release()
        log("sensitivity done")
    if args.what in ("table", "all"):
        table = sp.build_table(works, LOAD_GRID, log=log)
        result["table"] = json.loads(table.to_json())
        result["validation"] = sp.validate(table, works, args.heldout, log=log)
        v = result["validation"]
        log(f"held-out slowdown prediction: n={v['n']} nearest: mean {v['mean_rel_err']:.3f} p90 "
            f"{v['p90_rel_err']:.3f}; interpolated: mean {v['interp_mean_rel_err']:.3f} p90 {v['interp_p90_rel_err']:.3f}")
    with open(args.out, "w") as f:
        json.dump(result, f)
    log(f"wrote {args.out}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
