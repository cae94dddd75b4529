"""Spatial-sharing reference: CU shares and the interference factor (test
infrastructure only; see the package docstring for who may import it).

The paper gives colocated operators disjoint SM shares through separate
streams (Section 2.1, "Sensitivity to SM Core Allocation") and models their
mutual slowdown with one empirical factor per operator pair (Section 4.4,
"Interference Model", Eq. 5): I = T~_v(b, p) / T_v(b, p), the latency of v
while co-running over its latency alone at the same share p.  Factors are
stored on a 5 % grid of shares, a query takes the nearest profiled grid point,
and a three-way colocation is approximated by the product of the pairwise
factors.  (`multilinear` is the interpolating alternative to the nearest
point, over the same grid.)

On MI355X a share is a set of compute units named by a stream's CU mask.  The
library lays a share out evenly over the 8 XCDs (each XCD has its own L2 and
receives every 8th workgroup): position i of the balanced order is slot
i // X of XCD i % X, and a share is a range of positions.  The hardware names
CU (XCD x, slot s) by mask bit s * X + x when the mask is interleaved over the
XCDs and x * (N / X) + s when it is blocked by XCD.

Parity status: `cu_mask` is pinned by brute-force properties (popcount,
per-XCD balance, disjoint complementary shares); `corun_summary` by a worked
example and by invariants; `nearest` by exhaustive comparison; `interference`
and `three_way` by the identities they must satisfy; `multilinear` by
exactness on multilinear functions and at grid points.  None is "parity
unpinned".
"""
from __future__ import annotations

import math

import numpy as np


def balanced_positions(num_cus: int, num_xcds: int, first: int, count: int):
    """(xcd, slot) of the positions [first, first + count) of the balanced order."""
    assert num_cus % num_xcds == 0 and 0 <= first and first + count <= num_cus and count >= 1
    return [(i % num_xcds, i // num_xcds) for i in range(first, first + count)]


def mask_bit(num_cus: int, num_xcds: int, interleaved: bool, xcd: int, slot: int) -> int:
    """The CU-mask bit of CU `slot` of XCD `xcd` under the given mapping."""
    per = num_cus // num_xcds
    return slot * num_xcds + xcd if interleaved else xcd * per + slot


def cu_mask(num_cus: int, num_xcds: int, interleaved: bool, first: int, count: int):
    """The mask of a share as a list of uint32 words (bit n of word n // 32)."""
    words = [0] * ((num_cus + 31) // 32)
    for x, s in balanced_positions(num_cus, num_xcds, first, count):
        b = mask_bit(num_cus, num_xcds, interleaved, x, s)
        words[b // 32] |= 1 << (b % 32)
    return words


def mask_bits(words):
    """The set bits of a list of uint32 words."""
    return [32 * w + j for w, v in enumerate(words) for j in range(32) if (v >> j) & 1]


def median(values) -> float:
    """Median with linear interpolation between the two middle values; 0 for none."""
    v = np.sort(np.asarray(values, dtype=np.float64))
    if v.size == 0:
        return 0.0
    pos = 0.5 * (v.size - 1)
    lo, hi = math.floor(pos), math.ceil(pos)
    return float(v[lo] + (v[hi] - v[lo]) * (pos - lo))


def interference(t_co: float, t_iso: float) -> float:
    """Eq. 5: co-run latency over isolated latency at the same share."""
    return t_co / t_iso


def corun_summary(a_start, a_end, b_start, b_end, a_iso, b_iso):
    """T, T~ and I of both operators from the raw launch times of one co-run:
    T is the median isolated launch, T~ the median of the launches that lie
    wholly inside the other operator's active span (its first launch's start
    to its last launch's end)."""
    a_start, a_end, b_start, b_end = (np.asarray(x, np.float64) for x in (a_start, a_end, b_start, b_end))

    def inside(s, e, lo, hi):
        keep = (s >= lo) & (e <= hi)
        return (e - s)[keep]

    co_a = inside(a_start, a_end, b_start[0], b_end[-1])
    co_b = inside(b_start, b_end, a_start[0], a_end[-1])
    ta, tb = median(a_iso), median(b_iso)
    out = {"overlap_a": int(co_a.size), "overlap_b": int(co_b.size), "a_iso_us": ta, "b_iso_us": tb,
           "a_co_us": median(co_a), "b_co_us": median(co_b)}
    out["interference_a"] = interference(out["a_co_us"], ta) if co_a.size else 0.0
    out["interference_b"] = interference(out["b_co_us"], tb) if co_b.size else 0.0
    return out


def nearest(grid, x: float, log: bool = False):
    """The grid point nearest x (in log space if `log`); ties go to the lower point."""
    best, best_d = None, None
    for g in sorted(grid):
        d = abs(math.log(g) - math.log(x)) if log else abs(g - x)
        if best_d is None or d < best_d - 1e-12:
            best, best_d = g, d
    return best


def multilinear(axes, logs, values, point) -> float:
    """Multilinear interpolation of values(corner) on a rectilinear grid:
    axes[i] the sorted grid points of axis i, logs[i] whether axis i is
    interpolated in log space, point clamped to the grid's range per axis.
    Written as the weighted sum over the 2^d corners of the enclosing cell."""
    per_axis = []
    for grid, lg, x in zip(axes, logs, point):
        g = sorted(grid)
        t = (lambda z: math.log(z)) if lg else (lambda z: z)
        x = min(max(x, g[0]), g[-1])
        j = max(i for i in range(len(g)) if g[i] <= x)
        if j == len(g) - 1:
            per_axis.append([(g[j], 1.0)])
        else:
            w = (t(x) - t(g[j])) / (t(g[j + 1]) - t(g[j]))
            per_axis.append([(g[j], 1.0 - w), (g[j + 1], w)])
    total = 0.0
    stack = [((), 1.0)]
    for choices in per_axis:
        stack = [(c + (g,), w * wg) for c, w in stack for g, wg in choices]
    for corner, w in stack:
        if w:
            total += w * values(corner)
    return total


def three_way(i_vu: float, i_vw: float) -> float:
    """Three-way colocation of v with u and w: the product of the pair factors."""
    return i_vu * i_vw
