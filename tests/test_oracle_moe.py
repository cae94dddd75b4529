"""Pins of the MoE oracle: routing against brute force and the softmax of a
library routine, the fused expert MLP against the dense SwiGLU MLP (one
expert) and against invariants that a dropped weight, a swapped projection
or a wrong expert index would break; plus planted mistakes."""
import types

import numpy as np
import pytest
from scipy.special import softmax as sp_softmax

import oracle
from oracle import moe as om


def _problem(seed, T=7, H=12, F=5, E=4):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(T, H))
    w1 = rng.normal(size=(E, 2 * F, H)) * 0.3
    w2 = rng.normal(size=(E, H, F)) * 0.3
    return x, w1, w2


def check_routing(impl):
    rng = np.random.default_rng(1)
    lg = rng.normal(size=(40, 6)).astype(np.float32)
    for k in (1, 2, 3, 6):
        ids, w = impl.topk_route(lg, k, False)
        assert ids.shape == (40, k)
        # the same set as the best k-subset, listed by decreasing logit
        assert np.array_equal(np.sort(ids, 1), om.topk_route_bruteforce(lg, k))
        assert np.all(np.diff(np.take_along_axis(lg, ids, 1), axis=1) <= 0)
        p = sp_softmax(lg.astype(np.float64), axis=1)
        assert np.allclose(w, np.take_along_axis(p, ids, 1), rtol=1e-12, atol=0)
        ids_r, w_r = impl.topk_route(lg, k, True)
        assert np.array_equal(ids_r, ids) and np.allclose(w_r.sum(1), 1.0)
        assert np.allclose(w_r, w / w.sum(1, keepdims=True))
    # equal logits: the lower expert index first
    ids, _ = impl.topk_route(np.array([[0.5, 2.0, 0.5, 2.0, 0.5]], np.float32), 3, False)
    assert ids.tolist() == [[1, 3, 0]]


def check_fused_moe(impl):
    x, w1, w2 = _problem(2)
    T, H = x.shape
    E, F2, _ = w1.shape
    F = F2 // 2
    # one expert, k = 1, weight 1: the dense SwiGLU MLP of the layer operators
    dense = oracle.linear(oracle.swiglu(oracle.linear(x, w1[0])), w2[0])
    got = impl.fused_moe(x, w1[:1], w2[:1], np.zeros((T, 1), int), np.ones((T, 1)))
    assert np.allclose(got, dense, rtol=1e-12, atol=1e-12)
    # hand example: H = 2, F = 1; gate row (1, 0), up row (0, 2), W2 column (1, -1)
    x1 = np.array([[1.0, 3.0]])
    w1h = np.array([[[1.0, 0.0], [0.0, 2.0]]])
    w2h = np.array([[[1.0], [-1.0]]])
    a = 1.0 / (1.0 + np.exp(-1.0)) * 6.0                  # silu(1) * 6
    assert np.allclose(impl.fused_moe(x1, w1h, w2h, [[0]], [[0.5]]), [[0.5 * a, -0.5 * a]], rtol=1e-14)
    rng = np.random.default_rng(3)
    ids = rng.integers(0, E, size=(T, 2))
    wts = rng.uniform(0.1, 1.0, size=(T, 2))
    base = impl.fused_moe(x, w1, w2, ids, wts)
    # linear in the routing weights
    assert np.allclose(impl.fused_moe(x, w1, w2, ids, 3.0 * wts), 3.0 * base, rtol=1e-12, atol=1e-12)
    # relabelling the experts together with their weights changes nothing
    perm = rng.permutation(E)
    inv = np.argsort(perm)
    assert np.allclose(impl.fused_moe(x, w1[perm], w2[perm], inv[ids], wts), base, rtol=1e-12, atol=1e-12)
    # two routes to one expert equal one route with the summed weight
    dup = impl.fused_moe(x, w1, w2, np.stack([ids[:, 0], ids[:, 0]], 1), np.stack([wts[:, 0], wts[:, 1]], 1))
    one = impl.fused_moe(x, w1, w2, ids[:, :1], (wts[:, 0] + wts[:, 1])[:, None])
    assert np.allclose(dup, one, rtol=1e-12, atol=1e-12)
    # each output row depends on its own token only
    x2 = x.copy()
    x2[0] += 1.0
    moved = impl.fused_moe(x2, w1, w2, ids, wts)
    assert np.allclose(moved[1:], base[1:], rtol=0, atol=0) and not np.allclose(moved[0], base[0])
    # the sum over slots equals the per-slot expert MLPs, expert by expert
    per = sum(wts[:, j:j + 1] * np.stack([om.expert_mlp(x[t:t + 1], w1[ids[t, j]], w2[ids[t, j]])[0]
                                          for t in range(T)]) for j in range(2))
    assert np.allclose(base, per, rtol=1e-12, atol=1e-12)
    # the gate half is the one under the SiLU: swapping the halves changes the result
    sw = np.concatenate([w1[:, F:], w1[:, :F]], axis=1)
    assert not np.allclose(impl.fused_moe(x, sw, w2, ids, wts), base)


def test_routing():
    check_routing(om)


def test_fused_moe():
    check_fused_moe(om)


def test_expert_without_tokens_is_skipped():
    x, w1, w2 = _problem(4, E=5)
    ids = np.full((x.shape[0], 1), 2)
    w2n = w2.copy()
    w2n[[0, 1, 3, 4]] = np.nan  # never read
    assert np.all(np.isfinite(om.fused_moe(x, w1, w2n, ids, np.ones((x.shape[0], 1)))))


# ------------------------------------------------------------ planted errors --
def _mutant(**over):
    m = types.SimpleNamespace(**{n: getattr(om, n) for n in dir(om) if not n.startswith("_")})
    for k, v in over.items():
        setattr(m, k, v)
    return m


def _route(order_fn=None, weights_fn=None):
    def f(logits, k, renormalize):
        lg = np.asarray(logits)
        T, E = lg.shape
        ids, w = np.zeros((T, k), np.int64), np.zeros((T, k))
        for t in range(T):
            order = order_fn(lg[t], E, k) if order_fn else sorted(range(E), key=lambda e: (-float(lg[t, e]), e))[:k]
            z = lg[t].astype(np.float64)
            p = weights_fn(z) if weights_fn else np.exp(z - z.max()) / np.exp(z - z.max()).sum()
            ids[t], w[t] = order, p[order]
            if renormalize:
                w[t] /= w[t].sum()
        return ids, w
    return f


def _moe_variant(gate_up_swapped=False, drop_weight=False, w2_transposed_experts=False):
    def f(x, w1, w2, topk_ids, topk_weights):
        x = np.asarray(x, float)
        T, H = x.shape
        E = np.asarray(w1).shape[0]
        F = np.asarray(w1).shape[1] // 2
        out = np.zeros((T, H))
        for t in range(T):
            for j, e in enumerate(np.asarray(topk_ids)[t]):
                h = np.asarray(w1[e], float) @ x[t]
                g, u = (h[F:], h[:F]) if gate_up_swapped else (h[:F], h[F:])
                e2 = (E - 1 - e) if w2_transposed_experts else e
                y = np.asarray(w2[e2], float) @ (g / (1 + np.exp(-g)) * u)
                out[t] += (1.0 if drop_weight else float(np.asarray(topk_weights)[t, j])) * y
        return out
    return f


MUTANTS = {
    "route_smallest_logits": (check_routing, dict(topk_route=_route(
        order_fn=lambda row, E, k: sorted(range(E), key=lambda e: (float(row[e]), e))[:k]))),
    "route_ties_upper_index": (check_routing, dict(topk_route=_route(
        order_fn=lambda row, E, k: sorted(range(E), key=lambda e: (-float(row[e]), -e))[:k]))),
    "route_weights_unnormalized_exp": (check_routing, dict(topk_route=_route(weights_fn=lambda z: np.exp(z)))),
    "moe_gate_up_swapped": (check_fused_moe, dict(fused_moe=_moe_variant(gate_up_swapped=True))),
    "moe_routing_weight_dropped": (check_fused_moe, dict(fused_moe=_moe_variant(drop_weight=True))),
    "moe_wrong_down_expert": (check_fused_moe, dict(fused_moe=_moe_variant(w2_transposed_experts=True))),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    check, over = MUTANTS[name]
    with pytest.raises(AssertionError):
        check(_mutant(**over))
