"""Benchmark of the per-operator decoder-layer forward on one MI355X.

One step = one pass of every operator of the hot path over one batch:
  prefill layer of a Llama-3-8B-shaped model on a ragged batch of 16 prompts
  (8871 tokens): RMSNorm -> QKV linear -> causal GQA prefill attention -> O
  linear -> RMSNorm -> gate-up linear -> SwiGLU -> down linear,
  then decode attention for 256 sequences over a paged KV cache (contexts
  uniform in [128, 8192], 4.5 GB of K/V).
Every operator is timed on its own with device events on the stream it runs
on.  `value` = prefill tokens per second of the whole step (the decode
attention is inside the step time, so this is conservative).

Prints one JSON line.  --gpus above 1 is refused (this build runs on one GPU).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15     # dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12      # HBM3E, B/s
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.json")
KERNEL_SOURCES = {"gemm_bf16_w4_kernel": "paper_2608_13499_amd/csrc/k_gemm.hip",
                  "gemm_bf16_kernel": "paper_2608_13499_amd/csrc/k_gemm.hip",
                  "rope_kernel": "paper_2608_13499_amd/csrc/k_layer_ops.hip",
                  "cache_write_kernel": "paper_2608_13499_amd/csrc/k_layer_ops.hip",
                  "add_rmsnorm_kernel": "paper_2608_13499_amd/csrc/k_layer_ops.hip",
                  "attn_prefill_bf16_kernel": "paper_2608_13499_amd/csrc/k_attn_prefill.hip",
                  "attn_decode_split_kernel": "paper_2608_13499_amd/csrc/k_attn_decode.hip",
                  "attn_decode_combine_kernel": "paper_2608_13499_amd/csrc/k_attn_decode.hip",
                  "rmsnorm_kernel": "paper_2608_13499_amd/csrc/k_norm_act.hip",
                  "swiglu_kernel": "paper_2608_13499_amd/csrc/k_norm_act.hip"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_sha(kernel: str) -> str:
    """Hash of the kernel's source file with comments and whitespace removed,
    so that only a change of the code itself invalidates its counters."""
    import re
    with open(os.path.join(ROOT, KERNEL_SOURCES[kernel])) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = "".join(src.split())
    return hashlib.sha256(src.encode()).hexdigest()[:16]


def gpu_state():
    """Shader clock, memory clock and package power of GPU 0 as rocm-smi
    reports them (read from a child process; None where it reports nothing)."""
    import re
    import shutil
    import subprocess
    try:
        # rocm-smi is a Python script: run it with this interpreter, so that
        # the child starts it directly (no #!/usr/bin/env hop that would exec
        # a second program).
        script = os.path.realpath(shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi")
        r = subprocess.run([sys.executable, script, "-d", "0", "--showclocks", "--showpower", "--json"],
                           capture_output=True, text=True, timeout=30)
        card = next(iter(json.loads(r.stdout).values()))
    except Exception as ex:  # noqa: BLE001 - the record is informative only
        return {"error": f"rocm-smi: {type(ex).__name__}"}

    def num(pred):
        for k, v in card.items():
            if pred(k.lower()):
                m = re.search(r"[-+]?\d+(\.\d+)?", str(v))
                if m:
                    return float(m.group(0))
        return None
    return {"sclk_mhz": num(lambda k: k.startswith("sclk clock speed")),
            "mclk_mhz": num(lambda k: k.startswith("mclk clock speed")),
            "power_w": num(lambda k: "power" in k and "(w)" in k)}


def measured_traffic(op: str, kernel: str):
    """HBM bytes per launch of `op` (FETCH_SIZE + WRITE_SIZE, calibrated) from
    the committed counter summary, or None when the kernel's source changed
    since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    e = t.get("ops", {}).get(op)
    if not e or e.get("kernel") != kernel or e.get("source_sha") != source_sha(kernel):
        return None
    return e.get("bytes_per_launch")


class Layer:
    """Preallocated operands of one step (inputs resident in HBM): the prefill
    layer of `pc` and, when `dc` is given, decode attention of `dc`."""

    def __init__(self, ops, wl, torch, pc=None, dc=None):
        self.ops, self.torch = ops, torch
        self.pc = pc or wl.C2
        self.dc = dc
        pc = self.pc
        self.p = wl.prefill_layer_inputs(pc)
        self.d = wl.decode_inputs(dc) if dc is not None else None
        M, H, F = self.p["M"], pc.hidden, pc.ffn
        Hq, Hkv, D = pc.n_q_heads, pc.n_kv_heads, pc.head_dim
        bf = torch.bfloat16
        e = lambda *s: torch.empty(*s, dtype=bf, device="cuda")
        self.h1, self.qkv, self.attn = e(M, H), e(M, pc.qkv_out), e(M, Hq, D)
        self.o, self.h2, self.gu, self.act, self.y = e(M, H), e(M, H), e(M, 2 * F), e(M, F), e(M, H)
        self.q = self.qkv[:, : Hq * D].view(M, Hq, D)
        self.k = self.qkv[:, Hq * D:(Hq + Hkv) * D].view(M, Hkv, D)
        self.v = self.qkv[:, (Hq + Hkv) * D:].view(M, Hkv, D)
        self.scale = 1.0 / math.sqrt(D)
        self.max_seqlen = int(self.p["lengths"].max())
        # one workspace for the linears' split partials, sized for the largest
        self.lws = torch.empty(max(16, max(ops.opscale_linear_workspace_size(M, N, K)
                                           for N, K in ((pc.qkv_out, H), (H, Hq * D), (2 * F, H), (H, F)))),
                               dtype=torch.uint8, device="cuda")
        self.names = ["rmsnorm_1", "qkv_linear", "attn_prefill", "o_linear", "rmsnorm_2",
                      "gate_up_linear", "swiglu", "down_linear"]
        dd = self.d
        if dd is not None:
            B = len(dd["context_lens_host"])
            self.ws = torch.empty(ops.opscale_attn_decode_workspace_size(B, dc.n_q_heads, dc.head_dim,
                                                                        dd["max_context_len"]),
                                  dtype=torch.uint8, device="cuda")
            self.dout = torch.empty_like(dd["q"])
            self.names.append("attn_decode")

    def step(self, events=None):
        ops, p, d = self.ops, self.p, self.d
        eps = self.pc.eps

        def mark(i):
            if events is not None:
                events[i].record()
        ws = self.lws
        mark(0)
        ops.opscale_rmsnorm(p["x"], p["w_norm1"], y=self.h1, eps=eps); mark(1)
        ops.opscale_linear(self.h1, p["w_qkv"], y=self.qkv, workspace=ws); mark(2)
        ops.opscale_attn_prefill(self.q, self.k, self.v, p["cu_seqlens"], self.max_seqlen, self.scale,
                                 True, out=self.attn); mark(3)
        ops.opscale_linear(self.attn.view(self.p["M"], -1), p["w_o"], y=self.o, workspace=ws); mark(4)
        ops.opscale_rmsnorm(self.o, p["w_norm2"], y=self.h2, eps=eps); mark(5)
        ops.opscale_linear(self.h2, p["w_gate_up"], y=self.gu, workspace=ws); mark(6)
        ops.opscale_swiglu(self.gu, out=self.act); mark(7)
        ops.opscale_linear(self.act, p["w_down"], y=self.y, workspace=ws); mark(8)
        if d is not None:
            ops.opscale_attn_decode(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["context_lens"],
                                    d["max_context_len"], self.scale, workspace=self.ws, out=self.dout); mark(9)

    def step_descs(self):
        """(name, descriptor) of each operator of the step, on the step's own buffers."""
        ops, p, d = self.ops, self.p, self.d
        eps = self.pc.eps
        ws = self.lws
        out = [
            ("rmsnorm_1", ops.desc_rmsnorm(p["x"], p["w_norm1"], self.h1, eps)),
            ("qkv_linear", ops.desc_linear(self.h1, p["w_qkv"], self.qkv, workspace=ws)),
            ("attn_prefill", ops.desc_attn_prefill(self.q, self.k, self.v, self.attn, p["cu_seqlens"],
                                                   self.max_seqlen, self.scale, True)),
            ("o_linear", ops.desc_linear(self.attn.view(self.p["M"], -1), p["w_o"], self.o, workspace=ws)),
            ("rmsnorm_2", ops.desc_rmsnorm(self.o, p["w_norm2"], self.h2, eps)),
            ("gate_up_linear", ops.desc_linear(self.h2, p["w_gate_up"], self.gu, workspace=ws)),
            ("swiglu", ops.desc_swiglu(self.gu, self.act)),
            ("down_linear", ops.desc_linear(self.act, p["w_down"], self.y, workspace=ws)),
        ]
        if d is not None:
            out.append(("attn_decode", ops.desc_attn_decode(d["q"], d["k_cache"], d["v_cache"], d["block_table"],
                                                            d["context_lens"], self.dout, d["max_context_len"],
                                                            self.scale, self.ws)))
        return out

    def setup_extras(self):
        """Operands of the operators around attention at the same shape: RoPE on
        the packed QKV output, the write of every token's k / v into a shuffled
        paged cache, and the residual add + norm of the O projection output."""
        import numpy as np
        import workloads as wl
        torch, pc = self.torch, self.pc
        lens = self.p["lengths"]
        bs = pc.block_size
        table, nb = wl.paged_cache_layout(lens, bs, wl.rng_for(pc, "block_table"))
        slots = np.concatenate([[table[b, j // bs] * bs + j % bs for j in range(L)] for b, L in enumerate(lens)])
        self.slots = torch.from_numpy(slots.astype(np.int32)).cuda()
        self.pos = torch.from_numpy(np.concatenate([np.arange(L) for L in lens]).astype(np.int32)).cuda()
        self.kc = torch.zeros(nb, bs, pc.n_kv_heads, pc.head_dim, dtype=torch.bfloat16, device="cuda")
        self.vc = torch.zeros_like(self.kc)
        self.res = wl.device_normal((self.p["M"], pc.hidden), pc.seed, "attn_out", "bf16")
        self.extra_names = ["rope", "reshape_and_cache", "add_rmsnorm"]

    def decode_linears(self):
        """The four projections of a decode step of the same layer at the
        decode batch (one row per sequence): descriptors for opscale_op_profile."""
        import workloads as wl
        pc, dc, ops = self.pc, self.dc, self.ops
        B = len(self.d["context_lens_host"])
        H, F, HqD = pc.hidden, pc.ffn, pc.n_q_heads * pc.head_dim
        bf = self.torch.bfloat16
        e = lambda *s_: self.torch.empty(*s_, dtype=bf, device="cuda")
        xs = {"h": wl.device_normal((B, H), dc.seed, "x", "bf16"),
              "attn": wl.device_normal((B, HqD), dc.seed, "attn_out", "bf16"),
              "act": wl.device_normal((B, F), dc.seed, "ffn_act", "bf16")}
        p = self.p
        plan = [("decode_qkv_linear", "h", p["w_qkv"]), ("decode_o_linear", "attn", p["w_o"]),
                ("decode_gate_up_linear", "h", p["w_gate_up"]), ("decode_down_linear", "act", p["w_down"])]
        self._dec_keep = [xs]
        out = []
        for name, xin, W in plan:
            y = e(B, W.shape[0])
            ws = self.torch.empty(max(16, ops.opscale_linear_workspace_size(B, W.shape[0], W.shape[1])),
                                  dtype=self.torch.uint8, device="cuda")
            self._dec_keep += [y, ws]
            out.append((name, ops.desc_linear(xs[xin], W, y, workspace=ws), B))
        return out

    def extra(self, i):
        ops, pc = self.ops, self.pc
        if i == 0:
            ops.opscale_rope(self.q, self.k, self.pos, pc.rope_theta)
        elif i == 1:
            ops.opscale_reshape_and_cache(self.k, self.v, self.kc, self.vc, self.slots)
        else:
            ops.opscale_add_rmsnorm(self.o, self.res, self.p["w_norm2"], y=self.h2, eps=pc.eps)

    def extra_work(self):
        pc = self.pc
        M, H = self.p["M"], pc.hidden
        Hq, Hkv, D = pc.n_q_heads, pc.n_kv_heads, pc.head_dim
        return {"rope": (3 * M * (Hq + Hkv) * D, 2 * 2 * M * (Hq + Hkv) * D + 4 * M, "hbm", M, "tokens/s"),
                "reshape_and_cache": (0, 4 * 2 * M * Hkv * D + 4 * M, "hbm", M, "tokens/s"),
                "add_rmsnorm": (5 * M * H, 2 * (4 * M * H + H), "hbm", M, "tokens/s")}

    def work(self):
        """Algorithmic (flops, bytes, bound, units, unit-name) per operator."""
        from_cost = _closed_forms()
        pc, dc = self.pc, self.dc
        M, H, F = self.p["M"], pc.hidden, pc.ffn
        Hq, Hkv, D = pc.n_q_heads, pc.n_kv_heads, pc.head_dim
        lens = self.p["lengths"]
        s = 2
        out = {
            "rmsnorm_1": (*from_cost["rmsnorm"](M, H, s), "hbm", M, "tokens/s"),
            "qkv_linear": (*from_cost["linear"](M, pc.qkv_out, H, s), "mfma", M, "tokens/s"),
            "attn_prefill": (*from_cost["attn_prefill"](lens, Hq, Hkv, D, s), "mfma", M, "tokens/s"),
            "o_linear": (*from_cost["linear"](M, H, Hq * D, s), "mfma", M, "tokens/s"),
            "rmsnorm_2": (*from_cost["rmsnorm"](M, H, s), "hbm", M, "tokens/s"),
            "gate_up_linear": (*from_cost["linear"](M, 2 * F, H, s), "mfma", M, "tokens/s"),
            "swiglu": (*from_cost["swiglu"](M, F, s), "hbm", M, "tokens/s"),
            "down_linear": (*from_cost["linear"](M, H, F, s), "mfma", M, "tokens/s"),
        }
        if self.d is not None:
            ctx = self.d["context_lens_host"]
            out["attn_decode"] = (*from_cost["attn_decode"](ctx, dc.n_q_heads, dc.n_kv_heads, dc.head_dim, s,
                                                            dc.block_size), "hbm", len(ctx), "seq/s")
        return out


def per_op_records(names, per_op_us, work):
    """tokens/s (seq/s), TFLOP/s, GB/s and roofline fraction of each operator
    from its average event-timed duration and its algorithmic work."""
    per_op = {}
    for nm in names:
        fl, by, bound, units, unit = work[nm]
        t_s = per_op_us[nm] * 1e-6
        att = min(PEAK_BF16, fl / by * PEAK_HBM)
        per_op[nm] = {"us": round(per_op_us[nm], 2), unit: round(units / t_s, 1),
                      "tflops": round(fl / t_s * 1e-12, 2), "gbps": round(by / t_s * 1e-9, 1),
                      "bound": bound, "roofline_frac": round((fl / t_s) / att, 4)}
    return per_op


def time_prefill_config(ops, wl, torch, cfg, steps: int, warmup: int):
    """The prefill layer of another configuration, operator by operator: each
    timed with device events on the stream it runs on, averaged over `steps`
    passes of the whole layer (inputs resident in HBM, as in the step)."""
    layer = Layer(ops, wl, torch, cfg, None)
    for _ in range(warmup):
        layer.step()
    torch.cuda.synchronize()
    n = len(layer.names)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n + 1)] for _ in range(steps)]
    t0 = time.perf_counter()
    for s_ in range(steps):
        layer.step(evs[s_])
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    us = {nm: sum(evs[s_][i].elapsed_time(evs[s_][i + 1]) for s_ in range(steps)) * 1e3 / steps
          for i, nm in enumerate(layer.names)}
    lens = layer.p["lengths"]
    M = layer.p["M"]
    rec = {"workload": f"{cfg.name} ({len(lens)} prompts, {M} tokens, lengths {int(lens.min())}-{int(lens.max())}, "
                       f"hidden {cfg.hidden}, {cfg.n_q_heads}/{cfg.n_kv_heads} heads x {cfg.head_dim}, FFN {cfg.ffn})",
           "tokens": M, "steps": steps, "ms_per_layer": round(ms, 4), "tokens/s": round(M / (ms * 1e-3), 1),
           "per_op": per_op_records(layer.names, us, layer.work())}
    del layer
    torch.cuda.empty_cache()
    return rec


def _closed_forms():
    """Algorithmic flop/byte counts of each operator (same closed forms as the
    library's timing struct; restated here so the benchmark's roofline does not
    depend on the library's own accounting)."""
    def rmsnorm(M, H, s):
        return 4 * M * H, s * (2 * M * H + H)

    def linear(M, N, K, s):
        return 2 * M * N * K, s * (M * K + N * K + M * N)

    def swiglu(M, F, s):
        return 6 * M * F, 3 * s * M * F

    def attn_prefill(lens, Hq, Hkv, D, s):
        T = int(sum(int(x) for x in lens))
        pairs = sum(int(x) * (int(x) + 1) // 2 for x in lens)
        return 4 * D * Hq * pairs, s * (2 * T * Hq * D + 2 * T * Hkv * D)

    def attn_decode(ctx, Hq, Hkv, D, s, bs):
        N = int(sum(int(x) for x in ctx))
        nb = sum((int(x) + bs - 1) // bs for x in ctx)
        return 4 * D * Hq * N, s * (2 * Hkv * D * N + 2 * len(ctx) * Hq * D) + 4 * (nb + len(ctx))
    return dict(rmsnorm=rmsnorm, linear=linear, swiglu=swiglu, attn_prefill=attn_prefill,
                attn_decode=attn_decode)


def _blas_info():
    """BLAS library and thread count NumPy uses (threadpoolctl)."""
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            return {"blas": f"{info[0].get('internal_api')} {info[0].get('version')}",
                    "threads": int(max(i.get("num_threads", 1) for i in info))}
    except Exception:  # noqa: BLE001 - informative only
        pass
    return {"blas": "unknown", "threads": len(os.sched_getaffinity(0))}


def cpu_baseline(budget_s: float = 20.0):
    """Time the CPU oracle as it stands (fp64 NumPy) on a bounded sample of the
    step's workload and scale it to the whole step: the per-row operators
    (both norms, the four full-width linears, SwiGLU) on `rows` token rows,
    scaled by M / rows; prefill attention on whole prompts, shortest first,
    scaled by the causal key-query pairs; decode attention on whole sequences
    of the decode batch, scaled by the cached keys.  value = prefill tokens of
    the step / the step's extrapolated time (the step includes decode
    attention, as on the GPU).  Reported as a baseline only."""
    import numpy as np

    import oracle
    import workloads as wl
    cfg, dcfg = wl.C2, wl.C3
    lens = wl.seq_lengths(cfg)
    M, H, F = int(lens.sum()), cfg.hidden, cfg.ffn
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    rows = 256
    g = lambda tag, shape, std=1.0, mean=0.0: wl.normal(wl.rng_for(cfg, tag), shape, std, mean).astype(np.float64)
    x = g("x", (rows, H))
    wn = g("w_norm", (H,), 0.02, 1.0)
    shapes = {"qkv": (cfg.qkv_out, H), "o": (H, Hq * D), "gate_up": (2 * F, H), "down": (H, F)}
    # Every output column of each linear is computed, 2048 columns per oracle
    # call, with one drawn 2048-row weight block per K (drawing and holding
    # the full fp64 weights costs more than the timed work; the values do not
    # change it).
    nblk = 2048
    Wb = {K: g("w_qkv" if K == H else "w_down", (nblk, K), 0.02) for K in {K for _, K in shapes.values()}}
    xs = {"qkv": x, "o": g("attn_out", (rows, Hq * D)), "gate_up": x, "down": g("ffn_act", (rows, F))}
    u = g("gate_up", (rows, 2 * F))
    t0 = time.perf_counter()
    oracle.rmsnorm(x, wn, cfg.eps)
    oracle.rmsnorm(x, wn, cfg.eps)
    for k, (N, K) in shapes.items():
        for _ in range(N // nblk):
            oracle.linear(xs[k], Wb[K])
    oracle.swiglu(u)
    per_row = (time.perf_counter() - t0) / rows
    del Wb
    order = np.argsort(lens)
    done_pairs, att_s, used = 0, 0.0, []
    for b in order:
        L = int(lens[b])
        q, k, v = g("q", (L, Hq, D)), g("k", (L, Hkv, D)), g("v", (L, Hkv, D))
        t0 = time.perf_counter()
        oracle.attn_prefill(q, k, v, [0, L], 1 / math.sqrt(D), True)
        att_s += time.perf_counter() - t0
        done_pairs += L * (L + 1) // 2
        used.append(L)
        if att_s > budget_s * 0.5:
            break
    all_pairs = int(sum(int(L) * (int(L) + 1) // 2 for L in lens))
    # decode attention: sequences of the decode batch in their drawn order,
    # each in a cache of its own pages (block table 0, 1, 2, ...)
    ctx = wl.seq_lengths(dcfg)
    bs = dcfg.block_size
    dec_s, dec_keys, dec_used = 0.0, 0, 0
    for n in ctx:
        n = int(n)
        nb = (n + bs - 1) // bs
        kc = g("k_cache", (nb, bs, dcfg.n_kv_heads, dcfg.head_dim))
        vc = g("v_cache", (nb, bs, dcfg.n_kv_heads, dcfg.head_dim))
        qd = g("q", (1, dcfg.n_q_heads, dcfg.head_dim))
        t0 = time.perf_counter()
        oracle.attn_decode(qd, kc, vc, np.arange(nb)[None, :], np.array([n]), 1 / math.sqrt(dcfg.head_dim))
        dec_s += time.perf_counter() - t0
        dec_keys += n
        dec_used += 1
        if dec_s > budget_s * 0.15:
            break
    total_s = per_row * M + att_s * all_pairs / done_pairs + dec_s * int(ctx.sum()) / dec_keys
    info = _blas_info()
    return {"value": M / total_s, "unit": "tokens/s", "cores": info["threads"], "kind": "oracle",
            "blas": info["blas"],
            "sample": f"fp64 NumPy oracle ({info['blas']}, {info['threads']} threads): both RMS Norms, the 4 "
                      f"full-width linears (in 2048-column calls) and SwiGLU on {rows} token rows; prefill attention on {len(used)} whole "
                      f"prompts (lengths {used}); decode attention on {dec_used} whole sequences of the decode "
                      f"batch ({dec_keys} keys); scaled to the step ({M} prefill tokens, {int(ctx.sum())} cached "
                      f"keys) by rows, causal key-query pairs and keys"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run one device copy of this many MiB before the steps (counter calibration)")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the step only (no isolated, extra-operator, configuration, peak or copy records)")
    ap.add_argument("--config", default=None,
                    help="time only this prefill configuration's layer, operator by operator (e.g. "
                         "llama70b_prefill_16k, llama8b_bursty_longctx) and print its record")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(f"bench.py runs on one GPU only (asked for {a.gpus}); multi-GPU sharding is not part of "
              "this build.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_13499_amd as ops
    import workloads as wl
    assert torch.cuda.is_available(), "no GPU"
    ops.load()
    torch.cuda.set_device(0)
    if a.config is not None:
        cfg = wl.CONFIGS[a.config]
        log(f"config {cfg.name} ...")
        print(json.dumps(time_prefill_config(ops, wl, torch, cfg, a.steps, a.warmup)), flush=True)
        return
    log("building inputs ...")
    layer = Layer(ops, wl, torch, wl.C2, wl.C3)
    torch.cuda.synchronize()
    if a.calibrate_copy_mib:
        src = torch.empty(a.calibrate_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    log("warmup ...")
    for _ in range(a.warmup):
        layer.step()
    torch.cuda.synchronize()
    n = len(layer.names)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n + 1)] for _ in range(a.steps)]
    state_before = gpu_state()
    log(f"timing {a.steps} steps ...")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(a.steps):
        layer.step(evs[s])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    state_after = gpu_state()
    ms_step = (t1 - t0) * 1e3 / a.steps
    per_op_us = {nm: sum(evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(a.steps)) * 1e3 / a.steps
                 for i, nm in enumerate(layer.names)}
    work = layer.work()
    per_op = per_op_records(layer.names, per_op_us, work)
    dom = max(layer.names, key=lambda nm: per_op_us[nm])
    fl, by, bound, _, _ = work[dom]
    kernel = {"mfma": "gemm_bf16_w4_kernel", "hbm": "rmsnorm_kernel"}[bound] if "linear" in dom or "norm" in dom else \
        {"attn_prefill": "attn_prefill_bf16_kernel", "attn_decode": "attn_decode_split_kernel",
         "swiglu": "swiglu_kernel"}[dom]
    t_dom = per_op_us[dom] * 1e-6
    if bound == "mfma":
        roof = {"bound": "mfma", "achieved": round(fl / t_dom * 1e-12, 2), "peak": PEAK_BF16 * 1e-12,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(by / t_dom * 1e-9, 1), "peak": PEAK_HBM * 1e-9, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom, kernel)
    roof["kernel"] = f"{kernel} ({dom})"
    roof["work_per_launch"] = {"flops": fl, "bytes": by}
    if a.no_extras:
        print(json.dumps({"metric": "per-operator prefill tokens/s + % of MFMA/HBM roofline, Llama-8B-shaped layer",
                          "value": round(layer.p["M"] / (ms_step * 1e-3), 1), "unit": "tokens/s",
                          "ms_per_step": round(ms_step, 4), "per_op": per_op, "roofline": roof}), flush=True)
        return
    # Each operator of the step alone on its stream: with a read of a 512 MiB
    # buffer between iterations (primary: weights and activations come from
    # HBM, not the 256 MB last-level cache) and warm, median / p10 / p90 of HIP
    # events, with the clocks before and after.
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    iso_iters = max(20, a.steps)
    isolated = {}
    for nm, desc in layer.step_descs():
        before = gpu_state()
        pf = ops.opscale_op_profile(desc, 5, iso_iters, flush)
        pw = ops.opscale_op_profile(desc, 5, iso_iters, None)
        after = gpu_state()
        isolated[nm] = {
            "flushed": {"us_median": round(pf.us_median, 2), "us_p10": round(pf.us_p10, 2),
                        "us_p90": round(pf.us_p90, 2), "roofline_frac": round(pf.roofline_frac, 4)},
            "warm": {"us_median": round(pw.us_median, 2), "us_p10": round(pw.us_p10, 2),
                     "us_p90": round(pw.us_p90, 2), "roofline_frac": round(pw.roofline_frac, 4)},
            "sclk_mhz": [before.get("sclk_mhz"), after.get("sclk_mhz")],
            "mclk_mhz": [before.get("mclk_mhz"), after.get("mclk_mhz")],
            "power_w": [before.get("power_w"), after.get("power_w")],
        }
    del flush
    # The operators around attention of a full layer (RoPE, cache write,
    # residual + norm), timed separately: they are not part of the step.
    layer.setup_extras()
    extra_ops = {}
    for i, nm in enumerate(layer.extra_names):
        for _ in range(a.warmup):
            layer.extra(i)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * a.steps)]
        for j in range(a.steps):
            ev[2 * j].record()
            layer.extra(i)
            ev[2 * j + 1].record()
        torch.cuda.synchronize()
        us = sum(ev[2 * j].elapsed_time(ev[2 * j + 1]) for j in range(a.steps)) * 1e3 / a.steps
        fl, by, bound, units, unit = layer.extra_work()[nm]
        t_s = us * 1e-6
        extra_ops[nm] = {"us": round(us, 2), unit: round(units / t_s, 1), "gbps": round(by / t_s * 1e-9, 1),
                         "bound": bound, "roofline_frac": round(by / t_s / PEAK_HBM, 4)}
    # The decode step's projections at the decode batch (256 rows), each timed
    # cold (after a read of 512 MB evicts L2 and the last-level cache: the
    # layer's weights were last read a whole model step earlier).
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    for nm, desc, B in layer.decode_linears():
        pr = ops.opscale_op_profile(desc, a.warmup, a.steps, flush)
        extra_ops[nm] = {"us": round(pr.us_median, 2), "tokens/s": round(B / (pr.us_median * 1e-6), 1),
                         "tflops": round(pr.tflops, 1), "gbps": round(pr.gbps, 1),
                         "bound": "mfma+hbm", "roofline_frac": round(pr.roofline_frac, 4)}
    # The mixture-of-experts FFN of the paper's MoE models, cold as above:
    # Mixtral-8x7B over the prefill batch's 8871 tokens, Qwen2-57B-A14B at a
    # 256-token decode batch (synthetic routing: N(0, 1) router logits).
    for mc in (wl.MOE_MIXTRAL_PREFILL, wl.MOE_QWEN_DECODE):
        H, F, E, k, T = mc.hidden, mc.ffn, mc.experts, mc.topk, mc.tokens
        w1 = wl.device_normal((E, 2 * F, H), mc.seed, "moe_w1", "bf16", std=0.02)
        w2 = wl.device_normal((E, H, F), mc.seed, "moe_w2", "bf16", std=0.02)
        xm = wl.device_normal((T, H), mc.seed, "x", "bf16")
        ids, wts = ops.opscale_moe_topk(wl.device_normal((T, E), mc.seed, "router", "f32"), k, True)
        om = torch.empty_like(xm)
        wsm = torch.empty(ops.opscale_fused_moe_workspace_size(T, H, F, E, k), dtype=torch.uint8, device="cuda")
        pr = ops.opscale_op_profile(ops.desc_fused_moe(xm, w1, w2, ids, wts, om, wsm), a.warmup, a.steps, flush)
        extra_ops[mc.name] = {"us": round(pr.us_median, 2), "tokens/s": round(T / (pr.us_median * 1e-6), 1),
                              "tflops": round(pr.tflops, 1), "gbps": round(pr.gbps, 1),
                              "bound": "mfma" if pr.bound == 0 else "hbm", "roofline_frac": round(pr.roofline_frac, 4)}
        del w1, w2, xm, ids, wts, om, wsm
    del flush
    # The 70B-shaped layer (16384 tokens) and the bursty long-context mix
    # (4 x 32768 + 64 short prompts), operator by operator.
    configs = {}
    for cfg, n in ((wl.C4, max(3, a.steps // 2)), (wl.C5, 3)):
        log(f"config {cfg.name} ...")
        configs[cfg.name] = time_prefill_config(ops, wl, torch, cfg, n, 1)
    # The copy ceiling of the memory-bound operators: a device copy of the
    # same bytes (read + write) from cold caches (after a 512 MiB read), the
    # bound for an operator that streams its operands once.
    log("copy ceiling ...")
    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    M_, H_, F_ = layer.p["M"], layer.pc.hidden, layer.pc.ffn
    copy_ceiling = {}
    for nm, nbytes in (("rmsnorm", 2 * (2 * M_ * H_ + H_)), ("add_rmsnorm", 2 * (4 * M_ * H_ + H_)),
                       ("swiglu", 3 * 2 * M_ * F_)):
        src = torch.empty(nbytes // 2, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        ts = []
        for i in range(13):
            flush.sum()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            dst.copy_(src)
            e1.record()
            torch.cuda.synchronize()
            if i >= 2:
                ts.append(e0.elapsed_time(e1) * 1e3)
        ts.sort()
        us = ts[len(ts) // 2]
        copy_ceiling[nm] = {"bytes": nbytes, "copy_us_median": round(us, 2),
                            "copy_gbps": round(nbytes / us * 1e-3, 1),
                            "copy_frac_of_spec": round(nbytes / us * 1e-3 / (PEAK_HBM * 1e-9), 4)}
        del src, dst
    del flush
    for nm, key in (("rmsnorm", "rmsnorm_1"), ("swiglu", "swiglu")):
        if key in isolated:
            copy_ceiling[nm]["op_us_flushed"] = isolated[key]["flushed"]["us_median"]
    # Peaks re-measured on this GPU (sustained clock, real data): the spec
    # peaks above stay the primary denominators.
    log("peak probes ...")
    big = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    big2 = torch.empty_like(big)
    meas = {"mfma_bf16_tflops": round(ops.opscale_probe_mfma(32768, 10), 1),
            "hbm_read_gbps": round(ops.opscale_probe_hbm(big, None, 5), 1),
            "hbm_copy_gbps": round(ops.opscale_probe_hbm(big, big2, 5), 1)}
    del big, big2
    meas["spec_bf16_tflops"], meas["spec_hbm_gbps"] = PEAK_BF16 * 1e-12, PEAK_HBM * 1e-9
    roof["frac_of_measured"] = round(roof["achieved"] / (meas["mfma_bf16_tflops"] if roof["bound"] == "mfma"
                                                         else meas["hbm_read_gbps"]), 4)
    for nm, rec in per_op.items():
        rec["frac_of_measured"] = round(rec["tflops"] / meas["mfma_bf16_tflops"] if rec["bound"] == "mfma"
                                        else rec["gbps"] / meas["hbm_read_gbps"], 4)
    M = layer.p["M"]
    out = {
        "metric": "per-operator prefill tokens/s + % of MFMA/HBM roofline, Llama-8B-shaped layer",
        "value": round(M / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{layer.pc.name} (16 prompts, {M} tokens, hidden 4096, 32/8 heads x 128, "
                               f"FFN 14336) + {layer.dc.name} attention (256 seqs, contexts U[128,8192])",
                   "global_batch": M, "seq_len": int(layer.p["lengths"].max()), "parallelism": "none"},
        "roofline": roof,
        "per_op": per_op,
        "extra_ops": extra_ops,
        "configs": configs,
        "isolated": isolated,
        "measured_peaks": meas,
        "copy_ceiling": copy_ceiling,
        "gpu_state": {"before": state_before, "after": state_after},
    }
    if not a.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
