"""Mixture-of-experts FFN reference: top-k routing and the fused expert MLP
(test infrastructure only; see the package docstring for who may import it).

The paper's MoE models (Qwen2-57B-A14B, Mixtral-8x7B; Table 3) replace the
dense MLP by a FusedMoE operator, which it characterizes as a linear,
compute-heavy operator that dominates at short sequences (Section 2.1;
Appendix D).  It does not print the operator's formula, so the functions
below are the standard definition of the two steps, in fp64 (readings in
READINGS and the design notes):

* routing: per token, the k experts with the largest router logits, weighted
  by the softmax of all E logits at those experts (optionally renormalized to
  sum to one over the k);
* expert MLP: for the token's row x, expert e computes
  W2[e] (silu(W1g[e] x) * (W1u[e] x)), with W1[e] = [W1g; W1u] of shape
  [2F, H] (gate rows first) and W2[e] of shape [H, F];
* output: the routing-weighted sum of the k experts' outputs.

Parity status: pinned in tests/test_oracle_moe.py by reduction to the dense
SwiGLU MLP (one expert, k = 1), by invariants (linearity in the routing
weights, joint relabelling of experts, merging of duplicate routes, token
independence, experts that receive no token) and, for routing, by brute
force over all k-subsets.  None is "parity unpinned".
"""
from __future__ import annotations

import itertools

import numpy as np

READINGS = {
    "topk_order": "the k selected experts are listed by decreasing logit; equal logits go to the "
                  "lower expert index first (the selection compares the fp32 logits as given).",
    "topk_weights": "weights are softmax(logits over all E experts) at the selected experts, then "
                    "optionally divided by their sum (renormalize).",
    "w1_layout": "W1[e] is [2F, H]: rows 0..F-1 the gate projection, rows F..2F-1 the up "
                 "projection (the layout of the dense gate-up linear).",
    "invalid_expert": "an expert id outside [0, E) contributes nothing to its token.",
}


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def topk_route(logits, k: int, renormalize: bool):
    """Top-k routing of each token (row of logits [T, E]): (ids [T, k] int,
    weights [T, k] float64)."""
    lg = np.asarray(logits)
    T, E = lg.shape
    ids = np.zeros((T, k), dtype=np.int64)
    w = np.zeros((T, k))
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-float(lg[t, e]), e))[:k]
        z = _f64(lg[t])
        p = np.exp(z - z.max())
        p = p / p.sum()
        ids[t] = order
        w[t] = p[order]
        if renormalize:
            w[t] = w[t] / w[t].sum()
    return ids, w


def topk_route_bruteforce(logits, k: int):
    """The k-subset with the largest logit sum, ties by the lexicographically
    smallest index tuple: the same set as the top k (a pin, small E only)."""
    lg = np.asarray(logits, dtype=np.float64)
    T, E = lg.shape
    out = []
    for t in range(T):
        best = max(itertools.combinations(range(E), k), key=lambda c: (sum(lg[t, list(c)]), [-i for i in c]))
        out.append(sorted(best))
    return np.asarray(out)


def silu(z):
    z = _f64(z)
    return z / (1.0 + np.exp(-z))


def expert_mlp(x, w1, w2):
    """One expert's SwiGLU MLP on rows x [n, H]: W2 (silu(W1g x) * (W1u x))."""
    x, w1, w2 = _f64(x), _f64(w1), _f64(w2)
    F = w1.shape[0] // 2
    h = x @ w1.T
    return (silu(h[:, :F]) * h[:, F:]) @ w2.T


def fused_moe(x, w1, w2, topk_ids, topk_weights):
    """out[t] = sum_j topk_weights[t, j] * expert_mlp(x[t], W1[e], W2[e]),
    e = topk_ids[t, j]; x [T, H], w1 [E, 2F, H], w2 [E, H, F]."""
    x = _f64(x)
    T, H = x.shape
    E = np.asarray(w1).shape[0]
    ids = np.asarray(topk_ids)
    wts = _f64(topk_weights)
    out = np.zeros((T, H))
    for e in range(E):
        rows, slots = np.nonzero(ids == e)
        if rows.size == 0:
            continue
        y = expert_mlp(x[rows], w1[e], w2[e])
        np.add.at(out, rows, wts[rows, slots][:, None] * y)
    return out
