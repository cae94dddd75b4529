"""Shared helpers of the GPU parity tests: input generation (through the
seeded `workloads` module), transfers, and the error metric.

Error metric: for each checked output row (a token row for norm / linear /
SwiGLU, a (token, head) row of D values for attention),
    e_row = max_j |gpu_j - ref_j| / max(max_j |ref_j|, 1e-30)
and a test passes when max_row e_row <= tol: 2e-2 for bf16 (bf16 inputs, fp32
accumulation, bf16 output) and 1e-5 for the fp32 path.  A pure elementwise
relative error is unbounded where the reference crosses zero, which is why the
row maximum is the denominator.
"""
from __future__ import annotations

import sys

import numpy as np

import workloads as wl

TOL = {"bf16": 2e-2, "f32": 1e-5}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if got.size == 0:
        return 0.0
    D = ref.shape[-1]
    g = got.reshape(-1, D)
    r = ref.reshape(-1, D)
    assert np.isfinite(g).all(), "non-finite GPU output"
    den = np.maximum(np.abs(r).max(axis=1), 1e-30)
    return float((np.abs(g - r).max(axis=1) / den).max())


def assert_close(got, ref, dtype: str, what: str = ""):
    e = row_rel_err(got, ref)
    say(f"  {what}: max row-relative error {e:.3e} (tol {TOL[dtype]:.0e})")
    assert e <= TOL[dtype], f"{what}: error {e:.3e} > {TOL[dtype]:.0e}"
    return e


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def gen(seed, tag, shape, dtype, std=1.0, mean=0.0):
    """Seeded normal tensor in `dtype` on the CPU (bf16-rounded once)."""
    return wl.as_dtype(wl.normal(wl.rng_for(seed, tag), shape, std, mean), dtype)


def gen_large(seed, tag, shape, dtype, std=1.0, chunk=1 << 26):
    """Same distribution as `gen` for big tensors, drawn in chunks straight into
    the target dtype to bound host memory.  (Different draws than `gen`.)"""
    import torch
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch_dtype(dtype))
    rng = wl.rng_for(seed, tag)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        a = rng.standard_normal(m, dtype=np.float32)
        if std != 1.0:
            a *= np.float32(std)
        out[s:s + m] = torch.from_numpy(a).to(out.dtype)
    return out.view(*shape)


def f64(t) -> np.ndarray:
    return wl.to_f64(t)


def cuda(t):
    return t.to("cuda")
