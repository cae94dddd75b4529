"""Pins of the spatial-sharing oracle (CU shares, the co-run summary of Eq. 5,
nearest-grid lookup, the three-way product), each against a worked example,
a library routine or a brute-force property, plus planted mistakes that the
checks must catch."""
import types

import numpy as np
import pytest

import oracle
from oracle import spatial as osp


def hw_xcd(num_cus, num_xcds, interleaved, bit):
    """Which XCD the hardware runs mask bit `bit` on, for the two mask layouts
    the library recognises (interleaved over the XCDs, or blocked by XCD)."""
    return bit % num_xcds if interleaved else bit // (num_cus // num_xcds)


def check_cu_mask(impl):
    # worked example: 16 CUs over 4 XCDs, the first 6 positions of the balanced
    # order are (x, s) = (0,0) (1,0) (2,0) (3,0) (0,1) (1,1)
    assert impl.cu_mask(16, 4, False, 0, 6) == [0x1133]   # bits x*4 + s: 0 4 8 12 1 5
    assert impl.cu_mask(16, 4, True, 0, 6) == [0x3F]      # bits s*4 + x: 0 .. 5
    for N, X in [(256, 8), (64, 4), (40, 8), (12, 3), (8, 1)]:
        for il in (False, True):
            full = osp.mask_bits(impl.cu_mask(N, X, il, 0, N))
            assert full == list(range(N)), (N, X, il)          # every CU exactly once
            # the first X positions hold one CU of every XCD
            assert sorted(hw_xcd(N, X, il, b) for b in osp.mask_bits(impl.cu_mask(N, X, il, 0, X))) == list(range(X))
            for k in sorted({1, X - 1, X, X + 1, N // 3, N // 2, N - 1} - {0}):
                if not 1 <= k <= N - 1:
                    continue
                a = osp.mask_bits(impl.cu_mask(N, X, il, 0, k))
                b = osp.mask_bits(impl.cu_mask(N, X, il, k, N - k))
                assert len(a) == k and len(b) == N - k
                assert not set(a) & set(b) and sorted(a + b) == list(range(N))
                for share in (a, b):
                    per = np.bincount([hw_xcd(N, X, il, x) for x in share], minlength=X)
                    assert per.max() - per.min() <= 1, (N, X, il, k, per)


def check_corun_summary(impl):
    # A: durations 10 12 8 15 5; B's span is [5, 48], so A's launches 2..4 lie
    # inside it ([10,22] [22,30] [30,45]); B's two launches lie inside A's [0, 50]
    r = impl.corun_summary([0, 10, 22, 30, 45], [10, 22, 30, 45, 50], [5, 25], [25, 48],
                           [9, 11, 10, 10], [20, 22, 18])
    assert (r["overlap_a"], r["overlap_b"]) == (3, 2)
    assert r["a_iso_us"] == 10.0 and r["b_iso_us"] == 20.0
    assert r["a_co_us"] == 12.0 and r["b_co_us"] == 21.5
    assert abs(r["interference_a"] - 1.2) < 1e-12 and abs(r["interference_b"] - 1.075) < 1e-12
    # an operator that runs exactly as fast as alone has I = 1
    s = np.arange(0, 100, 4.0)                               # 25 launches, [0, 4] ... [96, 100]
    r = impl.corun_summary(s, s + 4, [1.0], [99.0], [4.0] * 5, [98.0])
    assert r["interference_a"] == 1.0 and r["overlap_a"] == 23  # starts 4 ... 92 lie in [1, 99]
    # disjoint spans: nothing overlaps
    r = impl.corun_summary([0, 1], [1, 2], [10], [11], [1, 1], [1])
    assert r["overlap_a"] == r["overlap_b"] == 0 and r["interference_a"] == r["interference_b"] == 0.0


def check_median(impl):
    rng = np.random.default_rng(3)
    for n in (1, 2, 5, 8, 101):
        x = rng.normal(size=n)
        assert abs(impl.median(x) - float(np.median(x))) < 1e-12
    assert impl.median([]) == 0.0


def check_nearest(impl):
    assert impl.nearest([16, 256], 64) == 16                 # 48 vs 192 apart
    assert impl.nearest([16, 256], 100) == 16
    assert impl.nearest([16, 256], 100, log=True) == 256     # ln 6.25 vs ln 2.56
    assert impl.nearest([16, 256], 64, log=True) == 16       # tie in log space: the lower point
    assert impl.nearest([0.05, 0.10, 0.15], 0.125) == 0.10   # tie: the lower point
    grid = [0.05 * i for i in range(1, 20)]
    for g in grid:
        assert impl.nearest(grid, g) == g
    rng = np.random.default_rng(5)
    for x in rng.uniform(0.0, 1.0, 200):                     # brute force over the grid
        d = [abs(g - x) for g in grid]
        assert impl.nearest(grid, x) == grid[int(np.argmin(d))]


def check_factors(impl):
    assert impl.interference(12.0, 10.0) == pytest.approx(1.2)
    assert impl.interference(7.5, 7.5) == 1.0
    assert impl.three_way(1.2, 1.5) == pytest.approx(1.8)
    assert impl.three_way(1.3, 1.0) == 1.3


def check_multilinear(impl):
    import math
    axes = [(16, 64, 256), (512, 2048, 8192), (0.05, 0.10, 0.15, 0.20)]
    logs = (True, True, False)
    # exact for a function multilinear in (log a, log b, c) ...
    f = lambda a, b, c: 1.0 + 0.3 * math.log(a) - 0.2 * math.log(b) + 2.0 * c + 0.05 * math.log(a) * c
    rng = np.random.default_rng(9)
    for _ in range(200):
        pt = (math.exp(rng.uniform(math.log(16), math.log(256))), math.exp(rng.uniform(math.log(512), math.log(8192))),
              rng.uniform(0.05, 0.20))
        assert abs(impl.multilinear(axes, logs, lambda c: f(*c), pt) - f(*pt)) < 1e-12
    # ... equal to the table at grid points, clamped outside the grid
    vals = {c: rng.uniform(1, 2) for c in np.ndindex(3, 3, 4)}
    table = lambda c: vals[(axes[0].index(c[0]), axes[1].index(c[1]), axes[2].index(c[2]))]
    for i, j, k in vals:
        assert impl.multilinear(axes, logs, table, (axes[0][i], axes[1][j], axes[2][k])) == vals[(i, j, k)]
    assert impl.multilinear(axes, logs, table, (1, 10 ** 6, 0.5)) == vals[(0, 2, 3)]
    # the log axis splits the cell at the geometric, not the arithmetic, midpoint
    one = [(16, 256)], (True,)
    assert abs(impl.multilinear(*one, lambda c: float(c[0] == 256), (64,)) - 0.5) < 1e-12


def test_cu_mask():
    check_cu_mask(osp)


def test_corun_summary():
    check_corun_summary(osp)


def test_median():
    check_median(osp)


def test_nearest():
    check_nearest(osp)


def test_factors():
    check_factors(osp)


def test_multilinear():
    check_multilinear(osp)


def test_exported_from_package():
    assert oracle.spatial is osp


# ------------------------------------------------------------ planted errors --
def _mutant(**over):
    m = types.SimpleNamespace(**{n: getattr(osp, n) for n in dir(osp) if not n.startswith("_")})
    for k, v in over.items():
        setattr(m, k, v)
    return m


def _mask_with(bit_fn=None, pos_fn=None):
    def f(N, X, il, first, count):
        words = [0] * ((N + 31) // 32)
        pos = pos_fn(N, X, first, count) if pos_fn else osp.balanced_positions(N, X, first, count)
        for x, s in pos:
            b = bit_fn(N, X, il, x, s) if bit_fn else osp.mask_bit(N, X, il, x, s)
            words[b // 32] |= 1 << (b % 32)
        return words
    return f


def _summary_any_overlap(a_s, a_e, b_s, b_e, ai, bi):
    a_s, a_e, b_s, b_e = (np.asarray(x, float) for x in (a_s, a_e, b_s, b_e))
    keep_a = (a_s < b_e[-1]) & (a_e > b_s[0])
    keep_b = (b_s < a_e[-1]) & (b_e > a_s[0])
    co_a, co_b = (a_e - a_s)[keep_a], (b_e - b_s)[keep_b]
    out = {"overlap_a": int(co_a.size), "overlap_b": int(co_b.size), "a_iso_us": osp.median(ai),
           "b_iso_us": osp.median(bi), "a_co_us": osp.median(co_a), "b_co_us": osp.median(co_b)}
    out["interference_a"] = out["a_co_us"] / out["a_iso_us"] if co_a.size else 0.0
    out["interference_b"] = out["b_co_us"] / out["b_iso_us"] if co_b.size else 0.0
    return out


def _summary_mean(*args):
    r = osp.corun_summary(*args)
    a_s, a_e, b_s, b_e = (np.asarray(x, float) for x in args[:4])
    keep = (a_s >= b_s[0]) & (a_e <= b_e[-1])
    if keep.any():
        r["a_co_us"] = float((a_e - a_s)[keep].mean())
        r["interference_a"] = r["a_co_us"] / r["a_iso_us"]
    return r


def _multilinear_linear_axes(axes, logs, values, point):
    return osp.multilinear(axes, [False] * len(axes), values, point)


def _multilinear_nearest(axes, logs, values, point):
    return values(tuple(osp.nearest(g, x, lg) for g, lg, x in zip(axes, logs, point)))


MUTANTS = {
    "multilinear_ignores_log": (check_multilinear, dict(multilinear=_multilinear_linear_axes)),
    "multilinear_is_nearest": (check_multilinear, dict(multilinear=_multilinear_nearest)),
    "mask_interleaved_bit_transposed": (check_cu_mask, dict(cu_mask=_mask_with(
        bit_fn=lambda N, X, il, x, s: x * X + s if il else x * (N // X) + s))),
    "mask_blocked_stride_is_xcds": (check_cu_mask, dict(cu_mask=_mask_with(
        bit_fn=lambda N, X, il, x, s: s * X + x if il else x * X + s))),
    "mask_positions_xcd_major": (check_cu_mask, dict(cu_mask=_mask_with(
        pos_fn=lambda N, X, first, count: [(i // (N // X), i % (N // X)) for i in range(first, first + count)]))),
    "corun_any_overlap_counts": (check_corun_summary, dict(corun_summary=_summary_any_overlap)),
    "corun_mean_not_median": (check_corun_summary, dict(corun_summary=_summary_mean)),
    "interference_inverted": (check_factors, dict(interference=lambda co, iso: iso / co)),
    "three_way_sum": (check_factors, dict(three_way=lambda a, b: a + b - 1.0)),
    "median_lower_middle": (check_median, dict(median=lambda v: float(np.sort(v)[(len(v) - 1) // 2]) if len(v) else 0.0)),
    "nearest_ignores_log": (check_nearest, dict(nearest=lambda grid, x, log=False: osp.nearest(grid, x))),
    "nearest_ties_upper": (check_nearest, dict(nearest=lambda grid, x, log=False: min(
        grid, key=lambda g: (abs(np.log(g) - np.log(x)) if log else abs(g - x), -g)))),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    check, over = MUTANTS[name]
    with pytest.raises(AssertionError):
        check(_mutant(**over))
