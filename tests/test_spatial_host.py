"""Host logic of spatial sharing (no GPU): the library's CU-mask builder and
the interference table against the oracle."""
import json
import math

import numpy as np
import pytest

import paper_2608_13499_amd as ops
from oracle import spatial as osp
from paper_2608_13499_amd import spatial as sp


@pytest.fixture(scope="module")
def lib():
    return ops.load()


def test_mask_build_matches_oracle(lib):
    rng = np.random.default_rng(11)
    cases = [(256, 8, il, f, c) for il in (0, 1) for f, c in ((0, 256), (0, 1), (0, 13), (13, 243), (0, 128),
                                                              (128, 128), (255, 1), (100, 37))]
    for _ in range(200):
        X = int(rng.choice([1, 2, 3, 4, 8]))
        N = X * int(rng.integers(1, 40))
        first = int(rng.integers(0, N))
        count = int(rng.integers(1, N - first + 1))
        cases.append((N, X, int(rng.integers(0, 2)), first, count))
    for N, X, il, first, count in cases:
        assert ops.opscale_cu_mask_build(N, X, il, first, count) == osp.cu_mask(N, X, bool(il), first, count), \
            (N, X, il, first, count)


@pytest.mark.parametrize("N,X,il,first,count,words", [
    (256, 8, 1, 0, 0, 8),      # empty share
    (256, 8, 1, 250, 13, 8),   # past the last CU
    (256, 8, 1, -1, 4, 8),     # negative first position
    (250, 8, 1, 0, 4, 8),      # CUs not a multiple of the XCDs
    (256, 8, 1, 0, 4, 7),      # too few words
    (0, 8, 1, 0, 1, 8),
])
def test_mask_build_rejects(lib, N, X, il, first, count, words):
    import ctypes
    buf = (ctypes.c_uint32 * max(1, words))()
    st = lib.opscale_cu_mask_build(N, X, il, first, count, buf, words)
    assert st == ops.OPSCALE_ERR_INVALID_ARG
    assert lib.opscale_last_error()


def test_mask_build_clears_extra_words(lib):
    import ctypes
    buf = (ctypes.c_uint32 * 10)(*([0xFFFFFFFF] * 10))
    assert lib.opscale_cu_mask_build(64, 4, 1, 0, 5, buf, 10) == ops.OPSCALE_OK
    assert list(buf)[2:] == [0] * 8 and list(buf)[:2] == osp.cu_mask(64, 4, True, 0, 5)


def test_stream_create_rejects_empty_mask(lib):
    import ctypes
    buf = (ctypes.c_uint32 * 8)()
    h = ctypes.c_void_p()
    assert lib.opscale_cu_stream_create(buf, 8, ctypes.byref(h)) == ops.OPSCALE_ERR_INVALID_ARG


def test_split_bounds():
    lay = sp.CULayout(256, 8, 1)
    assert lay.split(0.0) == 1 and lay.split(1.0) == 255 and lay.split(0.5) == 128
    assert lay.split(0.05) == 13 and lay.split(0.95) == 243


def test_snap_matches_oracle():
    rng = np.random.default_rng(2)
    for _ in range(300):
        grid = sorted(set(int(x) for x in rng.integers(1, 5000, rng.integers(1, 6))))
        x = float(rng.uniform(0.5, 6000))
        for log in (False, True):
            assert sp.snap(grid, x, log) == osp.nearest(grid, x, log)
    for x in np.linspace(0.0, 1.0, 101):
        assert sp.snap(sp.SHARE_GRID, float(x)) == osp.nearest(sp.SHARE_GRID, float(x))


def _random_table(seed=0):
    rng = np.random.default_rng(seed)
    loads = {"a": (16, 64, 256), "b": (512, 2048), "c": (100,)}
    t = sp.InterferenceTable(loads)
    for v in loads:
        for u in loads:
            for bv in loads[v]:
                for bu in loads[u]:
                    for p in t.shares:
                        t.put(v, bv, u, bu, p, 1.0 + rng.uniform(0, 0.8))
    return t


def test_lookup_snaps_to_the_oracle_grid_point():
    t = _random_table()
    rng = np.random.default_rng(4)
    for _ in range(300):
        v, u = rng.choice(["a", "b", "c"], 2)
        bv = float(math.exp(rng.uniform(math.log(4), math.log(5000))))
        bu = float(math.exp(rng.uniform(math.log(4), math.log(5000))))
        p = float(rng.uniform(0.0, 1.0))
        key = (v, osp.nearest(t.loads[v], bv, log=True), u, osp.nearest(t.loads[u], bu, log=True),
               round(osp.nearest(t.shares, p), 4))
        assert t.lookup(v, bv, u, bu, p) == t.entries[key]


def test_interpolation_matches_oracle():
    t = _random_table(3)
    rng = np.random.default_rng(6)
    for _ in range(300):
        v, u = rng.choice(["a", "b", "c"], 2)
        bv = float(math.exp(rng.uniform(math.log(4), math.log(5000))))
        bu = float(math.exp(rng.uniform(math.log(4), math.log(5000))))
        p = float(rng.uniform(0.0, 1.0))
        ref = osp.multilinear([t.loads[v], t.loads[u], t.shares], (True, True, False),
                              lambda c: t.entries[(v, c[0], u, c[1], round(c[2], 4))], (bv, bu, p))
        assert t.interpolate(v, bv, u, bu, p) == pytest.approx(ref, rel=1e-12)
    assert t.predict("a", 30, 0.33, [("b", 900), ("c", 100)], interpolate=True) == pytest.approx(
        osp.three_way(t.interpolate("a", 30, "b", 900, 0.33), t.interpolate("a", 30, "c", 100, 0.33)), rel=1e-15)


def test_three_way_is_the_product_of_pairs():
    t = _random_table(1)
    i_ab = t.lookup("a", 64, "b", 512, 0.3)
    i_ac = t.lookup("a", 64, "c", 100, 0.3)
    assert t.predict("a", 64, 0.3, [("b", 512)]) == i_ab
    assert t.predict("a", 64, 0.3, [("b", 512), ("c", 100)]) == pytest.approx(osp.three_way(i_ab, i_ac), rel=1e-15)


def test_table_json_round_trip():
    t = _random_table(2)
    t2 = sp.InterferenceTable.from_json(t.to_json())
    assert t2.entries == t.entries and t2.loads == t.loads and t2.shares == t.shares
    json.loads(t.to_json())


def test_relative_errors():
    e = sp.relative_errors([1.1, 0.9, 2.0], [1.0, 1.0, 2.0])
    assert np.allclose(e, [0.1, 0.1, 0.0])


def test_offgrid_load_in_range():
    rng = np.random.default_rng(0)
    for _ in range(100):
        b = sp._offgrid_load(rng, (16, 64, 256))
        assert 16 <= b <= 256 and b % 16 == 0


def test_workloads_cover_the_grid():
    w = sp.llama8b_workloads()
    assert set(w) == set(sp.LOAD_GRID)
    for k, wl in w.items():
        B, L = wl.shape(sp.LOAD_GRID[k][0])
        assert B >= 1 and L >= 1
