"""Pins for the CPU oracle: it is checked against things other than itself.

Each `check_*` function takes an implementation and raises AssertionError when
it disagrees with a brute-force loop, a hand-worked example under tests/golden,
a closed form, or an invariant of the operator's definition.  The plain tests
run every check on the oracle; the mutation tests plant plausible mistakes in
copies of the oracle (on the CPU) and require at least one check to catch each.
"""
import math
import os
import types

import numpy as np
import pytest

import oracle
from oracle import cost as ocost

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            out.append([np.array([float(t) for t in part.split()]) for part in line.split("|")])
    return out


# --------------------------------------------------------------- brute force --
def bf_linear(x, W, b=None):
    M, K = len(x), len(x[0])
    N = len(W)
    y = [[0.0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            acc = 0.0
            for k in range(K):
                acc += float(x[m][k]) * float(W[n][k])
            y[m][n] = acc + (float(b[n]) if b is not None else 0.0)
    return np.array(y)


def bf_rmsnorm(x, w, eps):
    out = []
    for row in x:
        ss = 0.0
        for v in row:
            ss += float(v) * float(v)
        r = math.sqrt(ss / len(row) + eps)
        out.append([float(v) / r * float(wj) for v, wj in zip(row, w)])
    return np.array(out)


def bf_attention_one(qv, keys, vals, scale):
    """softmax-weighted sum for one query, in plain Python floats."""
    s = [scale * sum(float(a) * float(b) for a, b in zip(qv, kk)) for kk in keys]
    m = max(s)
    e = [math.exp(t - m) for t in s]
    z = sum(e)
    D = len(vals[0])
    return [sum(e[j] / z * float(vals[j][d]) for j in range(len(keys))) for d in range(D)]


def bf_attn_prefill(q, k, v, cu, scale, causal):
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    out = np.zeros((T, Hq, D))
    for b in range(len(cu) - 1):
        s0, s1 = cu[b], cu[b + 1]
        for i in range(s1 - s0):
            for h in range(Hq):
                g = h // (Hq // Hkv)
                last = i if causal else (s1 - s0 - 1)
                keys = [k[s0 + j, g] for j in range(last + 1)]
                vals = [v[s0 + j, g] for j in range(last + 1)]
                out[s0 + i, h] = bf_attention_one(q[s0 + i, h], keys, vals, scale)
    return out


# -------------------------------------------------------------------- checks --
def check_linear(impl):
    rng = np.random.default_rng(1)
    for (M, N, K) in [(1, 1, 1), (3, 5, 7), (8, 4, 6), (2, 8, 8)]:
        x = rng.standard_normal((M, K))
        W = rng.standard_normal((N, K))
        b = rng.standard_normal(N)
        np.testing.assert_allclose(impl.linear(x, W), bf_linear(x, W), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(impl.linear(x, W, b), bf_linear(x, W, b), rtol=1e-12, atol=1e-12)
    for (M, K, N), x, W, y in [(tuple(int(t) for t in r[0]), r[1], r[2], r[3]) for r in _rows("linear_hand.txt")]:
        np.testing.assert_array_equal(impl.linear(x.reshape(M, K), W.reshape(N, K)), y.reshape(M, N))
    x = rng.standard_normal((5, 6))
    np.testing.assert_array_equal(impl.linear(x, np.eye(6)), x)


def check_rmsnorm(impl):
    rng = np.random.default_rng(2)
    for eps, x, w, y in _rows("rmsnorm_hand.txt"):
        np.testing.assert_allclose(impl.rmsnorm(x[None], w, float(eps[0]))[0], y, rtol=1e-15, atol=0)
    x = rng.standard_normal((6, 16))
    w = 1.0 + 0.02 * rng.standard_normal(16)
    np.testing.assert_allclose(impl.rmsnorm(x, w, 1e-5), bf_rmsnorm(x, w, 1e-5), rtol=1e-13)
    # unit RMS with unit gain: exactly 1 at eps = 0, 1/sqrt(1 + eps/mean(x^2)) otherwise
    y = impl.rmsnorm(x, np.ones(16), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-14)
    eps = 0.3
    y = impl.rmsnorm(x, np.ones(16), eps)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1 / np.sqrt(1 + eps / ms), rtol=1e-13)
    # constant row c: y = c / sqrt(c^2 + eps) * w
    c = -1.7
    np.testing.assert_allclose(impl.rmsnorm(np.full((1, 8), c), np.arange(1, 9.0), 0.5)[0],
                               c / math.sqrt(c * c + 0.5) * np.arange(1, 9.0), rtol=1e-14)


def check_swiglu(impl):
    (u, out), = _rows("swiglu_hand.txt")
    np.testing.assert_allclose(impl.swiglu(u[None])[0], out, rtol=1e-15, atol=1e-300)
    assert impl.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(impl.silu(np.array([1.0, -1.0])),
                               [1 / (1 + math.exp(-1)), -math.exp(-1) / (1 + math.exp(-1))], rtol=1e-15)
    rng = np.random.default_rng(3)
    g = rng.standard_normal((4, 9)) * 4
    np.testing.assert_allclose(impl.swiglu(np.concatenate([g, np.ones_like(g)], 1)), impl.silu(g), rtol=1e-15)
    np.testing.assert_allclose(impl.silu(g), [[v / (1 + math.exp(-v)) for v in row] for row in g], rtol=1e-14)
    # large negative gate: silu -> -0, no NaN
    assert np.isfinite(impl.silu(np.array([-1000.0, 1000.0]))).all()


def check_softmax(impl):
    rng = np.random.default_rng(4)
    s = rng.standard_normal((7, 13)) * 10
    p = impl.softmax(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(impl.softmax(s + 123.0), p, rtol=1e-12)
    for row, prow in zip(s, p):
        e = [math.exp(t - max(row)) for t in row]
        np.testing.assert_allclose(prow, [t / sum(e) for t in e], rtol=1e-13)


def check_attn_prefill(impl):
    # hand-worked two-key example, causal and not
    for causal, q, k, v, o in _rows("attn_two_keys.txt"):
        sh = (2, 1, 2)
        got = impl.attn_prefill(q.reshape(sh), k.reshape(sh), v.reshape(sh), [0, 2], 1.0, bool(causal[0]))
        np.testing.assert_allclose(got.reshape(-1), o, rtol=1e-14, atol=1e-14)
    rng = np.random.default_rng(5)
    # brute force on tiny ragged GQA batches, causal and not
    lens = [3, 1, 5, 0, 2]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    for Hq, Hkv in [(4, 2), (2, 2), (3, 1)]:
        q = rng.standard_normal((T, Hq, 4))
        k = rng.standard_normal((T, Hkv, 4))
        v = rng.standard_normal((T, Hkv, 4))
        for causal in (True, False):
            np.testing.assert_allclose(impl.attn_prefill(q, k, v, cu, 0.7, causal),
                                       bf_attn_prefill(q, k, v, cu, 0.7, causal), rtol=1e-12, atol=1e-12)
    # single-key attention returns V exactly
    q = rng.standard_normal((1, 2, 8))
    k = rng.standard_normal((1, 1, 8))
    v = rng.standard_normal((1, 1, 8))
    out = impl.attn_prefill(q, k, v, [0, 1], 0.3, True)
    assert np.array_equal(out[0, 0], v[0, 0]) and np.array_equal(out[0, 1], v[0, 0])
    # all keys equal: causal output is the running mean of v
    L = 6
    q = rng.standard_normal((L, 1, 4))
    k = np.tile(rng.standard_normal((1, 1, 4)), (L, 1, 1))
    v = rng.standard_normal((L, 1, 4))
    out = impl.attn_prefill(q, k, v, [0, L], 0.5, True)
    np.testing.assert_allclose(out[:, 0], np.cumsum(v[:, 0], 0) / np.arange(1, L + 1)[:, None], rtol=1e-13)
    # causal: perturbing k, v at positions > i leaves rows <= i unchanged
    L = 9
    q = rng.standard_normal((L, 2, 8))
    k = rng.standard_normal((L, 1, 8))
    v = rng.standard_normal((L, 1, 8))
    base = impl.attn_prefill(q, k, v, [0, L], 0.4, True)
    k2, v2 = k.copy(), v.copy()
    k2[5:] += 3.0
    v2[5:] -= 2.0
    pert = impl.attn_prefill(q, k2, v2, [0, L], 0.4, True)
    assert np.array_equal(base[:5], pert[:5])
    assert not np.allclose(base[5:], pert[5:])
    # GQA == MHA with each KV head repeated over its group
    Hq, Hkv = 6, 2
    q = rng.standard_normal((L, Hq, 8))
    k = rng.standard_normal((L, Hkv, 8))
    v = rng.standard_normal((L, Hkv, 8))
    gqa = impl.attn_prefill(q, k, v, [0, L], 0.35, True)
    mha = impl.attn_prefill(q, np.repeat(k, Hq // Hkv, axis=1), np.repeat(v, Hq // Hkv, axis=1), [0, L], 0.35, True)
    np.testing.assert_allclose(gqa, mha, rtol=1e-14)
    # batch composition: a ragged batch equals independent per-prompt calls
    lens = [4, 7, 1]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    q = rng.standard_normal((T, 4, 8))
    k = rng.standard_normal((T, 2, 8))
    v = rng.standard_normal((T, 2, 8))
    full = impl.attn_prefill(q, k, v, cu, 0.35, True)
    for b in range(3):
        s0, s1 = cu[b], cu[b + 1]
        one = impl.attn_prefill(q[s0:s1], k[s0:s1], v[s0:s1], [0, s1 - s0], 0.35, True)
        np.testing.assert_allclose(full[s0:s1], one, rtol=1e-14)
    # row-sampled evaluation agrees with the full evaluation
    rows = [(0, 0), (3, 1), (4, 3), (10, 2), (11, 0)]
    np.testing.assert_allclose(impl.attn_prefill_rows(q, k, v, cu, rows, 0.35, True),
                               np.stack([full[t, h] for t, h in rows]), rtol=1e-13)
    fulln = impl.attn_prefill(q, k, v, cu, 0.35, False)
    np.testing.assert_allclose(impl.attn_prefill_rows(q, k, v, cu, rows, 0.35, False),
                               np.stack([fulln[t, h] for t, h in rows]), rtol=1e-13)


def check_attn_decode(impl):
    (bt, kc, vc, q, o), = _rows("decode_paged_hand.txt")
    got = impl.attn_decode(q.reshape(1, 1, 2), kc.reshape(3, 2, 1, 2), vc.reshape(3, 2, 1, 2),
                           bt.astype(np.int64).reshape(1, 2), np.array([3]), 1.0)
    np.testing.assert_allclose(got.reshape(-1), o, rtol=1e-14)
    rng = np.random.default_rng(6)
    bs, Hkv, Hq, D = 4, 2, 4, 8
    ctx = np.array([1, 5, 8, 0, 13])
    nblk = (ctx + bs - 1) // bs
    nb = int(nblk.sum()) + 3
    perm = rng.permutation(nb)
    table = np.zeros((len(ctx), int(nblk.max())), np.int64)
    pos = 0
    for b, n in enumerate(nblk):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    kc = rng.standard_normal((nb, bs, Hkv, D))
    vc = rng.standard_normal((nb, bs, Hkv, D))
    q = rng.standard_normal((len(ctx), Hq, D))
    out = impl.attn_decode(q, kc, vc, table, ctx, 0.3)
    # brute force gather through the block table, element by element
    for b, n in enumerate(ctx):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            if n == 0:
                assert np.all(out[b, h] == 0)
                continue
            keys = [kc[table[b, j // bs], j % bs, g] for j in range(n)]
            vals = [vc[table[b, j // bs], j % bs, g] for j in range(n)]
            np.testing.assert_allclose(out[b, h], bf_attention_one(q[b, h], keys, vals, 0.3), rtol=1e-12, atol=1e-13)
    # single cached key returns V exactly
    assert np.array_equal(out[0, 0], vc[table[0, 0], 0, 0])
    # relabelling physical blocks (and moving the data with them) changes nothing
    relabel = rng.permutation(nb)
    kc2 = np.empty_like(kc)
    vc2 = np.empty_like(vc)
    kc2[relabel] = kc
    vc2[relabel] = vc
    out2 = impl.attn_decode(q, kc2, vc2, relabel[table], ctx, 0.3)
    np.testing.assert_allclose(out2, out, rtol=1e-14)
    # decode over the first n tokens == last row of causal prefill over those n tokens
    n = 11
    kseq = rng.standard_normal((n, Hkv, D))
    vseq = rng.standard_normal((n, Hkv, D))
    qseq = rng.standard_normal((n, Hq, D))
    pre = impl.attn_prefill(qseq, kseq, vseq, [0, n], 0.25, True)
    nb = (n + bs - 1) // bs
    kc = np.zeros((nb, bs, Hkv, D))
    vc = np.zeros((nb, bs, Hkv, D))
    for j in range(n):
        kc[j // bs, j % bs] = kseq[j]
        vc[j // bs, j % bs] = vseq[j]
    dec = impl.attn_decode(qseq[n - 1:n], kc, vc, np.arange(nb)[None], np.array([n]), 0.25)
    np.testing.assert_allclose(dec[0], pre[n - 1], rtol=1e-13)


def check_rope(impl):
    rng = np.random.default_rng(7)
    T, H, D, theta = 6, 3, 16, 10000.0
    x = rng.standard_normal((T, H, D))
    pos = np.array([0, 1, 2, 7, 100, 33000])
    out = impl.rope(x, pos, theta)
    # position 0 is the identity
    assert np.array_equal(out[0], x[0])
    # unit vectors: e_i rotates into (cos a_i, sin a_i) on the pair (i, i + D/2)
    # with a_i = p * theta^(-2i/D); e_{i+D/2} into (-sin a_i, cos a_i)
    half = D // 2
    for i in range(half):
        for p_ in (1, 5, 1000):
            a = p_ * theta ** (-2.0 * i / D)
            e = np.zeros((1, 1, D))
            e[0, 0, i] = 1.0
            r = impl.rope(e, [p_], theta)[0, 0]
            want = np.zeros(D)
            want[i], want[i + half] = math.cos(a), math.sin(a)
            np.testing.assert_allclose(r, want, atol=1e-12)
            e = np.zeros((1, 1, D))
            e[0, 0, i + half] = 1.0
            r = impl.rope(e, [p_], theta)[0, 0]
            want = np.zeros(D)
            want[i], want[i + half] = -math.sin(a), math.cos(a)
            np.testing.assert_allclose(r, want, atol=1e-12)
    # a rotation: every pair keeps its length
    np.testing.assert_allclose(out[..., :half] ** 2 + out[..., half:] ** 2,
                               x[..., :half] ** 2 + x[..., half:] ** 2, rtol=1e-12)
    # the same map written as complex multiplication z * exp(i a)
    z = (x[..., :half] + 1j * x[..., half:]) * np.exp(1j * pos[:, None, None] * theta ** (-2.0 * np.arange(half) / D))
    np.testing.assert_allclose(out, np.concatenate([z.real, z.imag], -1), atol=1e-11)
    # rotations compose: rope(rope(x, m), n) == rope(x, m + n)
    m, n = np.array([3, 40, 0, 9, 1, 2]), np.array([5, 1, 77, 0, 8, 1000])
    np.testing.assert_allclose(impl.rope(impl.rope(x, m, theta), n, theta), impl.rope(x, m + n, theta), atol=1e-11)
    # scores depend on the position difference only
    q, k = rng.standard_normal((1, 1, D)), rng.standard_normal((1, 1, D))
    for (mq, nk) in [(10, 3), (200, 190), (7, 7)]:
        lhs = float(np.sum(impl.rope(q, [mq], theta) * impl.rope(k, [nk], theta)))
        rhs = float(np.sum(impl.rope(q, [mq - nk], theta) * k))
        assert abs(lhs - rhs) < 1e-10 * (1 + abs(rhs))


def check_cache_write(impl):
    rng = np.random.default_rng(8)
    nb, bs, Hkv, D = 6, 4, 2, 3
    kc0 = rng.standard_normal((nb, bs, Hkv, D))
    vc0 = rng.standard_normal((nb, bs, Hkv, D))
    # one sequence of 7 tokens living in blocks (4, 1): slots follow the table
    table = np.array([4, 1])
    k = rng.standard_normal((9, Hkv, D))
    v = rng.standard_normal((9, Hkv, D))
    slots = np.array([table[j // bs] * bs + j % bs for j in range(7)] + [-1, nb * bs])  # two skipped
    kc, vc = impl.reshape_and_cache(k, v, kc0, vc0, slots)
    # reading the sequence back through the block table returns the new rows
    np.testing.assert_array_equal(oracle.gather_paged(kc, table, 7), k[:7])
    np.testing.assert_array_equal(oracle.gather_paged(vc, table, 7), v[:7])
    # every slot not written (including the last block's rows) is unchanged
    written = np.zeros((nb, bs), bool)
    for s_ in slots[:7]:
        written[s_ // bs, s_ % bs] = True
    np.testing.assert_array_equal(kc[~written], kc0[~written])
    np.testing.assert_array_equal(vc[~written], vc0[~written])
    # the inputs are not modified
    assert not np.shares_memory(kc, kc0)


def check_add_rmsnorm(impl):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((5, 12))
    res = rng.standard_normal((5, 12))
    w = 1 + 0.02 * rng.standard_normal(12)
    y, r = impl.add_rmsnorm(x, res, w, 1e-5)
    np.testing.assert_array_equal(r, x + res)
    # unit gain, eps 0: the normalized sum has RMS 1
    y1, _ = impl.add_rmsnorm(x, res, np.ones(12), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y1 * y1, -1)), 1.0, rtol=1e-13)
    # the sum, not x alone, is normalized: a constant sum c gives c / sqrt(c^2 + eps) * w
    c = 0.7
    yc, _ = impl.add_rmsnorm(np.full((1, 12), c) - res[:1], res[:1], w, 0.5)
    np.testing.assert_allclose(yc[0], c / math.sqrt(c * c + 0.5) * w, rtol=1e-12)
    # residual = -x: the sum is zero and so is the output (eps > 0)
    y0, r0 = impl.add_rmsnorm(x, -x, w, 1e-5)
    assert np.all(r0 == 0) and np.all(y0 == 0)


def check_layer(impl):
    """Prefill of L tokens then one decode step equals prefill of L + 1 tokens:
    RoPE positions, cache slots, attention and the residual path agree."""
    rng = np.random.default_rng(10)
    H, Hq, Hkv, D, F, eps, theta, bs = 16, 4, 2, 4, 24, 1e-5, 10000.0, 2
    p = {"w_norm1": 1 + 0.02 * rng.standard_normal(H), "w_qkv": 0.3 * rng.standard_normal(((Hq + 2 * Hkv) * D, H)),
         "w_o": 0.3 * rng.standard_normal((H, Hq * D)), "w_norm2": 1 + 0.02 * rng.standard_normal(H),
         "w_gate_up": 0.3 * rng.standard_normal((2 * F, H)), "w_down": 0.3 * rng.standard_normal((H, F))}
    lens = [5, 3]
    x_all = [rng.standard_normal((L + 1, H)) for L in lens]
    res_all = [rng.standard_normal((L + 1, H)) for L in lens]
    nb = 8
    table = np.array([[6, 1, 3], [0, 5, 2]])
    kc0, vc0 = np.zeros((nb, bs, Hkv, D)), np.zeros((nb, bs, Hkv, D))
    # prefill of the first L tokens of both sequences
    x = np.concatenate([a[:L] for a, L in zip(x_all, lens)])
    res = np.concatenate([a[:L] for a, L in zip(res_all, lens)])
    pos = np.concatenate([np.arange(L) for L in lens])
    slots = np.concatenate([[table[b, j // bs] * bs + j % bs for j in range(L)] for b, L in enumerate(lens)])
    cu = np.concatenate([[0], np.cumsum(lens)])
    pre = impl.decoder_layer_forward(x, res, p, pos, cu, Hq, Hkv, D, eps, theta, kc0, vc0, slots)
    # one decode step with token L of each sequence
    xd = np.stack([a[L] for a, L in zip(x_all, lens)])
    rd = np.stack([a[L] for a, L in zip(res_all, lens)])
    dec = impl.decoder_layer_decode(xd, rd, p, np.array(lens) + 1, table, Hq, Hkv, D, eps, theta,
                                    pre["k_cache"], pre["v_cache"])
    for b, L in enumerate(lens):
        full = impl.decoder_layer_forward(x_all[b], res_all[b], p, np.arange(L + 1), [0, L + 1], Hq, Hkv, D, eps,
                                          theta, kc0, vc0, [-1] * (L + 1))
        for key in ("y", "r2", "attn", "q", "k"):
            np.testing.assert_allclose(dec[key][b], full[key][L], rtol=1e-10, atol=1e-11)
    # the decode step wrote its k and v where the prefill of L + 1 tokens would have
    assert list(dec["slots"]) == [table[b, L // bs] * bs + L % bs for b, L in enumerate(lens)]
    # no residual means the input itself is the residual
    a = impl.decoder_layer_forward(x, None, p, pos, cu, Hq, Hkv, D, eps, theta, kc0, vc0, slots)
    b_ = impl.decoder_layer_forward(x, np.zeros_like(x), p, pos, cu, Hq, Hkv, D, eps, theta, kc0, vc0, slots)
    np.testing.assert_allclose(a["y"], b_["y"], rtol=1e-13)


def _kv(name):
    """A golden of `key value value ...` lines, as a dict of float arrays."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                key, *vals = line.split()
                out[key] = np.array([float(t) for t in vals])
    return out


def check_layer_golden(impl):
    """The two-token layer worked by hand: every intermediate, the written
    cache, the output and the carried residual (tests/golden/layer_two_tokens_hand.txt)."""
    g = _kv("layer_two_tokens_hand.txt")
    H, D, F = int(g["H"][0]), int(g["D"][0]), int(g["F"][0])
    Hq, Hkv = (int(t) for t in g["heads"])
    T = len(g["positions"])
    nb, bs = int(g["num_blocks"][0]), int(g["block_size"][0])
    p = {"w_norm1": g["w_norm1"], "w_norm2": g["w_norm2"],
         "w_qkv": g["w_qkv"].reshape((Hq + 2 * Hkv) * D, H), "w_o": g["w_o"].reshape(H, Hq * D),
         "w_gate_up": g["w_gate_up"].reshape(2 * F, H), "w_down": g["w_down"].reshape(H, F)}
    fill = np.full((nb, bs, Hkv, D), g["cache_fill"][0])
    out = impl.decoder_layer_forward(g["x"].reshape(T, H), g["residual"].reshape(T, H), p,
                                     g["positions"].astype(int), g["cu_seqlens"].astype(int), Hq, Hkv, D,
                                     float(g["eps"][0]), float(g["theta"][0]), fill, fill,
                                     g["slots"].astype(int))
    for key in ("h1", "q", "k", "v", "k_cache", "v_cache", "attn", "o", "r2", "h2", "act", "y"):
        np.testing.assert_allclose(np.asarray(out[key]).ravel(), g[key], rtol=1e-12, atol=1e-13,
                                   err_msg=key)


def check_cost(c):
    # causal visible pairs counted by a loop
    lens = [1, 2, 5, 0, 9]
    pairs = sum(1 for L in lens for i in range(L) for j in range(L) if j <= i)
    f, b = c.attn_prefill(lens, 4, 2, 8, 2, True)
    assert f == 4 * 8 * 4 * pairs
    T = sum(lens)
    assert b == 2 * (2 * T * 4 * 8 + 2 * T * 2 * 8)
    f, _ = c.attn_prefill(lens, 4, 2, 8, 2, False)
    assert f == 4 * 8 * 4 * sum(L * L for L in lens)
    assert c.linear(3, 5, 7, 2) == (2 * 3 * 5 * 7, 2 * (21 + 35 + 15))
    assert c.linear(3, 5, 7, 4, bias=True)[1] == 4 * (21 + 35 + 15 + 5)
    assert c.rmsnorm(4, 8, 2)[1] == 2 * (2 * 32 + 8)
    assert c.swiglu(4, 8, 2)[1] == 2 * 3 * 32
    ctx = [1, 16, 17, 0]
    f, b = c.attn_decode(ctx, 8, 2, 4, 2, 16)
    assert f == 4 * 4 * 8 * 34
    assert b == 2 * (2 * 2 * 4 * 34 + 2 * 4 * 8 * 4) + 4 * ((1 + 1 + 2 + 0) + 4)
    # rope: q and k elements read and written once, 3 flops per element (6 per pair)
    assert c.rope(5, 4, 2, 8, 2) == (3 * 5 * 6 * 8, 2 * 2 * 5 * 6 * 8 + 4 * 5)
    # cache write: k and v read and written, plus one int32 slot per token
    assert c.reshape_and_cache(5, 2, 8, 2) == (0, 4 * 2 * 5 * 2 * 8 + 4 * 5)
    # residual + norm: x, residual read; sum and output written; gain read once
    assert c.add_rmsnorm(4, 8, 2) == (5 * 32, 2 * (4 * 32 + 8))


CHECKS = [check_linear, check_rmsnorm, check_swiglu, check_softmax, check_attn_prefill, check_attn_decode,
          check_rope, check_cache_write, check_add_rmsnorm, check_layer, check_layer_golden]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_pinned(check):
    check(oracle)


def test_cost_closed_forms():
    check_cost(ocost)


# ------------------------------------------------------------ planted errors --
def _mutant(**overrides):
    m = types.SimpleNamespace(**{n: getattr(oracle, n) for n in dir(oracle) if not n.startswith("_")})
    for k, v in overrides.items():
        setattr(m, k, v)
    return m


def _mut_attn(kv_map=None, causal_strict=False, drop_scale=False, no_max=False):
    """A copy of the prefill definition with one planted mistake."""
    def f(q, k, v, cu, scale, causal=True):
        q, k, v = np.asarray(q, float), np.asarray(k, float), np.asarray(v, float)
        T, Hq, D = q.shape
        Hkv = k.shape[1]
        out = np.zeros((T, Hq, D))
        for b in range(len(cu) - 1):
            s0, s1 = int(cu[b]), int(cu[b + 1])
            L = s1 - s0
            if L == 0:
                continue
            vis = np.tril(np.ones((L, L), bool), -1 if causal_strict else 0) if causal else np.ones((L, L), bool)
            vis[0, 0] = True
            for h in range(Hq):
                g = kv_map(h, Hq, Hkv) if kv_map else h // (Hq // Hkv)
                s = (1.0 if drop_scale else scale) * (q[s0:s1, h] @ k[s0:s1, g].T)
                s = np.where(vis, s, -np.inf)
                e = np.exp(s - (0 if no_max else s.max(-1, keepdims=True)))
                out[s0:s1, h] = (e / e.sum(-1, keepdims=True)) @ v[s0:s1, g]
        return out
    return f


def _mut_rope(interleaved=False, sign=1.0, exp_scale=2.0):
    def f(x, positions, theta):
        x = np.asarray(x, float)
        D = x.shape[-1]
        half = D // 2
        ang = np.asarray(positions, float)[:, None] * float(theta) ** (-exp_scale * np.arange(half) / D)
        c, s = np.cos(ang)[:, None, :], sign * np.sin(ang)[:, None, :]
        if interleaved:
            a, b = x[..., 0::2], x[..., 1::2]
            out = np.empty_like(x)
            out[..., 0::2], out[..., 1::2] = a * c - b * s, b * c + a * s
            return out
        a, b = x[..., :half], x[..., half:]
        return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)
    return f


def _mut_cache(skip_check=True, swap=False):
    def f(k, v, kc, vc, slots):
        kc, vc = np.array(kc, float), np.array(vc, float)
        nb, bs = kc.shape[:2]
        for t, s_ in enumerate(slots):
            if skip_check and not 0 <= s_ < nb * bs:
                continue
            if not skip_check and s_ >= nb * bs:
                continue
            blk, off = (s_ % nb, s_ // nb) if swap else (s_ // bs, s_ % bs)
            kc[blk, off], vc[blk, off] = k[t], v[t]
        return kc, vc
    return f


def _mut_layer_decode_pos(x, res, p, ctx, bt, Hq, Hkv, D, eps, theta, kc, vc):
    """decode step that rotates the new token by position context_len instead of
    context_len - 1 (and writes it one slot later)."""
    return oracle.decoder_layer_decode(x, res, p, np.asarray(ctx) + 1, np.concatenate([bt, bt[:, -1:]], 1),
                                       Hq, Hkv, D, eps, theta, kc, vc)


def _mut_layer(norm2_without_residual=False, gate_up_fed_h1=False, carry_r1=False, first_norm_of_x=False,
               rope_q_only=False, cache_before_rope=False, attend_unrotated=False, rope_v=False):
    """A copy of the prefill layer dataflow with one planted wiring mistake."""
    def f(x, residual, p, positions, cu, Hq, Hkv, D, eps, theta, kc, vc, slots):
        T = x.shape[0]
        x = np.asarray(x, float)
        r1 = x if residual is None else x + residual
        h1 = oracle.rmsnorm(x if first_norm_of_x else r1, p["w_norm1"], eps)
        qkv = oracle.linear(h1, p["w_qkv"])
        q0 = qkv[:, : Hq * D].reshape(T, Hq, D)
        k0 = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
        v = qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D)
        q = oracle.rope(q0, positions, theta)
        k = k0 if rope_q_only else oracle.rope(k0, positions, theta)
        if rope_v:
            v = oracle.rope(v, positions, theta)
        kc2, vc2 = oracle.reshape_and_cache(k0 if cache_before_rope else k, v, kc, vc, slots)
        a = oracle.attn_prefill(q0 if attend_unrotated else q, k0 if attend_unrotated else k, v, cu,
                                1.0 / np.sqrt(D), causal=True)
        o = oracle.linear(a.reshape(T, Hq * D), p["w_o"])
        r2 = r1 if carry_r1 else o + r1
        h2 = oracle.rmsnorm(o if norm2_without_residual else o + r1, p["w_norm2"], eps)
        gu = oracle.linear(h1 if gate_up_fed_h1 else h2, p["w_gate_up"])
        act = oracle.swiglu(gu)
        y = oracle.linear(act, p["w_down"])
        return {"h1": h1, "r1": r1, "qkv": qkv, "q": q, "k": k, "v": v, "attn": a, "o": o, "h2": h2, "r2": r2,
                "gate_up": gu, "act": act, "y": y, "k_cache": kc2, "v_cache": vc2}
    return f


def _mut_layer_decode_attends_first(x, res, p, ctx, bt, Hq, Hkv, D, eps, theta, kc, vc):
    """decode step whose attention reads the cache before its own k and v are
    written to it."""
    out = oracle.decoder_layer_decode(x, res, p, ctx, bt, Hq, Hkv, D, eps, theta, kc, vc)
    a = oracle.attn_decode(out["q"], kc, vc, bt, ctx, 1.0 / np.sqrt(D))
    B = x.shape[0]
    o = oracle.linear(a.reshape(B, Hq * D), p["w_o"])
    h2, r2 = oracle.add_rmsnorm(o, out["r1"], p["w_norm2"], eps)
    y = oracle.linear(oracle.swiglu(oracle.linear(h2, p["w_gate_up"])), p["w_down"])
    return dict(out, attn=a, o=o, h2=h2, r2=r2, y=y)


MUTANTS = {
    "linear_k_reversed": (check_linear, dict(linear=lambda x, W, b=None: np.asarray(x, float) @ np.asarray(W, float)[:, ::-1].T + (0 if b is None else b))),
    "linear_bias_dropped": (check_linear, dict(linear=lambda x, W, b=None: np.asarray(x, float) @ np.asarray(W, float).T)),
    "rmsnorm_eps_outside": (check_rmsnorm, dict(rmsnorm=lambda x, w, eps: np.asarray(x) / (np.sqrt(np.mean(np.asarray(x) ** 2, -1, keepdims=True)) + eps) * w)),
    "rmsnorm_sum_not_mean": (check_rmsnorm, dict(rmsnorm=lambda x, w, eps: np.asarray(x) / np.sqrt(np.sum(np.asarray(x) ** 2, -1, keepdims=True) + eps) * w)),
    "rmsnorm_one_plus_w": (check_rmsnorm, dict(rmsnorm=lambda x, w, eps: oracle.rmsnorm(x, 1 + np.asarray(w, float), eps))),
    "swiglu_halves_swapped": (check_swiglu, dict(swiglu=lambda u: oracle.silu(np.asarray(u)[:, np.asarray(u).shape[1] // 2:]) * np.asarray(u)[:, : np.asarray(u).shape[1] // 2])),
    "silu_sign": (check_swiglu, dict(silu=lambda z: np.asarray(z, float) / (1 + np.exp(np.asarray(z, float))),
                                     swiglu=lambda u: (lambda z: z / (1 + np.exp(z)))(np.asarray(u, float)[:, : np.asarray(u).shape[1] // 2]) * np.asarray(u, float)[:, np.asarray(u).shape[1] // 2:])),
    "softmax_no_normalize": (check_softmax, dict(softmax=lambda s, axis=-1: np.exp(np.asarray(s) - np.max(s, axis=axis, keepdims=True)))),
    "attn_gqa_modulo": (check_attn_prefill, dict(attn_prefill=_mut_attn(kv_map=lambda h, Hq, Hkv: h % Hkv))),
    "attn_causal_strict": (check_attn_prefill, dict(attn_prefill=_mut_attn(causal_strict=True))),
    "attn_scale_dropped": (check_attn_prefill, dict(attn_prefill=_mut_attn(drop_scale=True))),
    "decode_slot_index": (check_attn_decode, dict(attn_decode=lambda q, kc, vc, bt, n, scale: oracle.attn_decode(q, kc[:, ::-1], vc[:, ::-1], bt, n, scale))),
    "decode_gqa_modulo": (check_attn_decode, dict(attn_decode=lambda q, kc, vc, bt, n, scale: oracle.attn_decode(q, np.asarray(kc)[:, :, ::-1], np.asarray(vc)[:, :, ::-1], bt, n, scale))),
    "rope_interleaved_pairs": (check_rope, dict(rope=_mut_rope(interleaved=True))),
    "rope_sign": (check_rope, dict(rope=_mut_rope(sign=-1.0))),
    "rope_exponent": (check_rope, dict(rope=_mut_rope(exp_scale=1.0))),
    "rope_position_off_by_one": (check_rope, dict(rope=lambda x, pos, th: oracle.rope(x, np.asarray(pos) + 1, th))),
    "cache_negative_slot_wraps": (check_cache_write, dict(reshape_and_cache=_mut_cache(skip_check=False))),
    "cache_block_offset_swapped": (check_cache_write, dict(reshape_and_cache=_mut_cache(swap=True))),
    "add_rmsnorm_norms_x": (check_add_rmsnorm, dict(add_rmsnorm=lambda x, r, w, eps: (oracle.rmsnorm(x, w, eps), np.asarray(x) + r))),
    "layer_decode_position_is_len": (check_layer, dict(decoder_layer_decode=_mut_layer_decode_pos)),
    "layer_decode_attends_before_cache_write": (check_layer, dict(decoder_layer_decode=_mut_layer_decode_attends_first)),
    "layer_norm2_without_residual": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(norm2_without_residual=True))),
    "layer_gate_up_fed_h1": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(gate_up_fed_h1=True))),
    "layer_carries_r1": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(carry_r1=True))),
    "layer_first_norm_of_x": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(first_norm_of_x=True))),
    "layer_rope_q_only": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(rope_q_only=True))),
    "layer_cache_before_rope": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(cache_before_rope=True))),
    "layer_attends_unrotated": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(attend_unrotated=True))),
    "layer_rope_on_v": (check_layer_golden, dict(decoder_layer_forward=_mut_layer(rope_v=True))),
}


def test_layer_copy_without_a_mistake_passes():
    """The mutant layer with no mistake planted matches the golden, so each
    wiring mutant fails for its planted mistake alone."""
    check_layer_golden(_mutant(decoder_layer_forward=_mut_layer()))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    check, over = MUTANTS[name]
    with pytest.raises(AssertionError):
        check(_mutant(**over))


@pytest.mark.parametrize("name,mut", [
    ("causal_pairs_strict", dict(attn_prefill=lambda L, Hq, Hkv, D, s, causal=True: (4 * D * Hq * int(sum(l * (l - 1) // 2 for l in L)), 0))),
    ("rope_q_only", dict(rope=lambda T, Hq, Hkv, D, s: (3 * T * Hq * D, 2 * s * T * Hq * D + 4 * T))),
    ("decode_blocks_floor", dict(attn_decode=lambda n, Hq, Hkv, D, s, bs: (4 * D * Hq * sum(n), s * (2 * Hkv * D * sum(n) + 2 * len(n) * Hq * D) + 4 * (sum(x // bs for x in n) + len(n))))),
])
def test_planted_cost_mistake_is_caught(name, mut):
    c = types.SimpleNamespace(**{k: getattr(ocost, k) for k in ("linear", "rmsnorm", "swiglu", "attn_prefill", "attn_decode",
                                                                "rope", "reshape_and_cache", "add_rmsnorm")})
    for k, v in mut.items():
        setattr(c, k, v)
    with pytest.raises(AssertionError):
        check_cost(c)
