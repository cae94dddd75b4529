"""ctypes binding of libopscale (include/opscale.h).

Argument marshalling only: every operator runs in the library's HIP kernels.
PyTorch supplies device memory and the current HIP stream.  The functions keep
the C names; tensors are passed instead of raw pointers, and sizes are taken
from the tensor shapes.  A missing library or a failed call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libopscale.so")

OPSCALE_OK, OPSCALE_ERR_INVALID_ARG, OPSCALE_ERR_UNSUPPORTED, OPSCALE_ERR_WORKSPACE, OPSCALE_ERR_HIP = range(5)
OPSCALE_F32, OPSCALE_BF16 = 0, 1
(OP_RMSNORM, OP_LINEAR, OP_SWIGLU, OP_ATTN_PREFILL, OP_ATTN_DECODE, OP_ROPE, OP_RESHAPE_AND_CACHE,
 OP_ADD_RMSNORM, OP_FUSED_MOE) = range(9)
(TUNE_GEMM_TILE, TUNE_GEMM_SKINNY, TUNE_GEMM_SPLITK, TUNE_GEMM_TAIL, TUNE_SKINNY_NG, TUNE_PREFILL_SCHEDULE,
 TUNE_MOE_FUSE, TUNE_GEMM_DECODE) = range(8)
TUNE_AUTO = -1

c_i32, c_i64, c_f32, c_f64, c_vp, c_sz = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                          ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t)


class OpscaleError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"opscale status {status}: {message}")
        self.status = status


class Timing(ctypes.Structure):
    _fields_ = [("elapsed_us", c_f32), ("alg_flops", c_f64), ("alg_bytes", c_f64)]


class _RmsnormArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("w", c_vp), ("y", c_vp), ("M", c_i64), ("H", c_i64), ("eps", c_f32)]


class _LinearArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("W", c_vp), ("bias", c_vp), ("y", c_vp), ("M", c_i64), ("N", c_i64), ("K", c_i64),
                ("workspace", c_vp), ("workspace_bytes", c_sz)]


class _SwigluArgs(ctypes.Structure):
    _fields_ = [("gate_up", c_vp), ("out", c_vp), ("M", c_i64), ("F", c_i64)]


class _PrefillArgs(ctypes.Structure):
    _fields_ = [("q", c_vp), ("k", c_vp), ("v", c_vp), ("q_row_stride", c_i64), ("kv_row_stride", c_i64),
                ("o", c_vp), ("cu_seqlens", c_vp), ("B", c_i32), ("total_tokens", c_i64),
                ("max_seqlen", c_i32), ("Hq", c_i32), ("Hkv", c_i32), ("D", c_i32), ("scale", c_f32),
                ("causal", c_i32)]


class _DecodeArgs(ctypes.Structure):
    _fields_ = [("q", c_vp), ("q_row_stride", c_i64), ("k_cache", c_vp), ("v_cache", c_vp), ("block_table", c_vp),
                ("context_lens", c_vp), ("o", c_vp), ("B", c_i32), ("Hq", c_i32), ("Hkv", c_i32),
                ("D", c_i32), ("block_size", c_i32), ("max_blocks_per_seq", c_i32), ("num_blocks", c_i64),
                ("max_context_len", c_i32), ("scale", c_f32), ("workspace", c_vp), ("workspace_bytes", c_sz)]


class _RopeArgs(ctypes.Structure):
    _fields_ = [("q", c_vp), ("k", c_vp), ("q_row_stride", c_i64), ("k_row_stride", c_i64), ("positions", c_vp),
                ("T", c_i64), ("Hq", c_i32), ("Hkv", c_i32), ("D", c_i32), ("theta", c_f64)]


class _CacheWriteArgs(ctypes.Structure):
    _fields_ = [("k", c_vp), ("v", c_vp), ("kv_row_stride", c_i64), ("k_cache", c_vp), ("v_cache", c_vp),
                ("slot_mapping", c_vp), ("T", c_i64), ("Hkv", c_i32), ("D", c_i32), ("block_size", c_i32),
                ("num_blocks", c_i64)]


class _AddRmsnormArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("residual", c_vp), ("w", c_vp), ("y", c_vp), ("M", c_i64), ("H", c_i64),
                ("eps", c_f32)]


class _FusedMoeArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("w1", c_vp), ("w2", c_vp), ("topk_ids", c_vp), ("topk_weights", c_vp), ("out", c_vp),
                ("T", c_i64), ("H", c_i32), ("F", c_i32), ("E", c_i32), ("topk", c_i32), ("workspace", c_vp),
                ("workspace_bytes", c_sz)]


class _OpUnion(ctypes.Union):
    _fields_ = [("rmsnorm", _RmsnormArgs), ("linear", _LinearArgs), ("swiglu", _SwigluArgs),
                ("attn_prefill", _PrefillArgs), ("attn_decode", _DecodeArgs), ("rope", _RopeArgs),
                ("reshape_and_cache", _CacheWriteArgs), ("add_rmsnorm", _AddRmsnormArgs),
                ("fused_moe", _FusedMoeArgs)]


class OpDesc(ctypes.Structure):
    _fields_ = [("op", c_i32), ("dt", c_i32), ("u", _OpUnion)]


class Profile(ctypes.Structure):
    _fields_ = [("iters", c_i32), ("us_median", c_f32), ("us_p10", c_f32), ("us_p90", c_f32),
                ("us_min", c_f32), ("us_mean", c_f32), ("alg_flops", c_f64), ("alg_bytes", c_f64),
                ("tflops", c_f64), ("gbps", c_f64), ("attainable_tflops", c_f64),
                ("roofline_frac", c_f64), ("bound", c_i32), ("weight_bytes", c_i64),
                ("transient_bytes", c_i64), ("io_bytes", c_i64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class Corun(ctypes.Structure):
    _fields_ = [("n_a", c_i32), ("n_b", c_i32), ("overlap_a", c_i32), ("overlap_b", c_i32),
                ("a_iso_us", c_f32), ("b_iso_us", c_f32), ("a_co_us", c_f32), ("b_co_us", c_f32),
                ("interference_a", c_f64), ("interference_b", c_f64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_PF = ctypes.POINTER(c_f32)


class _CorunTrace(ctypes.Structure):
    _fields_ = [("a_start", _PF), ("a_end", _PF), ("b_start", _PF), ("b_end", _PF), ("a_iso", _PF),
                ("b_iso", _PF)]


EXPORTS = {
    "opscale_version": (ctypes.c_char_p, []),
    "opscale_status_string": (ctypes.c_char_p, [c_i32]),
    "opscale_last_error": (ctypes.c_char_p, []),
    "opscale_rmsnorm": (c_i32, [c_vp, c_vp, c_vp, c_i64, c_i64, c_f32, c_i32, c_vp, ctypes.POINTER(Timing)]),
    "opscale_set_tuning": (c_i32, [c_i32, c_i32]),
    "opscale_get_tuning": (c_i32, [c_i32]),
    "opscale_linear_workspace_size": (c_sz, [c_i64, c_i64, c_i64, c_i32]),
    "opscale_linear": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64, c_i32, c_vp, c_sz, c_vp,
                               ctypes.POINTER(Timing)]),
    "opscale_swiglu": (c_i32, [c_vp, c_vp, c_i64, c_i64, c_i32, c_vp, ctypes.POINTER(Timing)]),
    "opscale_attn_prefill": (c_i32, [c_vp, c_vp, c_vp, c_i64, c_i64, c_vp, c_vp, c_i32, c_i64, c_i32,
                                     c_i32, c_i32, c_i32, c_f32, c_i32, c_i32, c_vp, ctypes.POINTER(Timing)]),
    "opscale_attn_decode_workspace_size": (c_sz, [c_i32, c_i32, c_i32, c_i32]),
    "opscale_attn_decode": (c_i32, [c_vp, c_i64, c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_i32,
                                    c_i32, c_i64, c_i32, c_f32, c_i32, c_vp, c_sz, c_vp,
                                    ctypes.POINTER(Timing)]),
    "opscale_attn_decode_noalloc": (c_i32, [c_vp, c_i64, c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32,
                                            c_i32, c_i32, c_i64, c_i32, c_f32, c_i32, c_vp]),
    "opscale_attn_decode_noalloc_max_bytes": (c_sz, []),
    "opscale_op_profile": (c_i32, [ctypes.POINTER(OpDesc), c_i32, c_i32, c_vp, c_sz, c_vp,
                                   ctypes.POINTER(Profile)]),
    "opscale_rope": (c_i32, [c_vp, c_vp, c_i64, c_i64, c_vp, c_i64, c_i32, c_i32, c_i32, ctypes.c_double, c_i32,
                             c_vp, ctypes.POINTER(Timing)]),
    "opscale_reshape_and_cache": (c_i32, [c_vp, c_vp, c_i64, c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i64,
                                          c_i32, c_vp, ctypes.POINTER(Timing)]),
    "opscale_add_rmsnorm": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_f32, c_i32, c_vp,
                                    ctypes.POINTER(Timing)]),
    "opscale_moe_topk": (c_i32, [c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_vp, ctypes.POINTER(Timing)]),
    "opscale_fused_moe_workspace_size": (c_sz, [c_i64, c_i32, c_i32, c_i32, c_i32]),
    "opscale_fused_moe": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_i32,
                                  c_vp, c_sz, c_vp, ctypes.POINTER(Timing)]),
    "opscale_cu_layout": (c_i32, [ctypes.POINTER(c_i32)] * 3),
    "opscale_cu_mask_build": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(ctypes.c_uint32), c_i32]),
    "opscale_cu_stream_create": (c_i32, [ctypes.POINTER(ctypes.c_uint32), c_i32, ctypes.POINTER(c_vp)]),
    "opscale_cu_stream_destroy": (c_i32, [c_vp]),
    "opscale_cu_stream_mask": (c_i32, [c_vp, ctypes.POINTER(ctypes.c_uint32), c_i32]),
    "opscale_cu_probe": (c_i32, [c_vp, c_vp, c_i32, c_i32]),
    "opscale_probe_mfma": (c_i32, [c_i64, c_i32, c_vp, ctypes.POINTER(c_f64)]),
    "opscale_probe_hbm": (c_i32, [c_vp, c_vp, c_sz, c_i32, c_vp, ctypes.POINTER(c_f64)]),
    "opscale_corun_profile": (c_i32, [ctypes.POINTER(OpDesc), c_vp, ctypes.POINTER(OpDesc), c_vp, c_i32, c_i32,
                                      c_f32, c_i32, ctypes.POINTER(_CorunTrace), ctypes.POINTER(Corun)]),
}

_lib = None


def load(path: Optional[str] = None):
    """Load libopscale.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise OpscaleError(-1, f"{path} is missing: build it with `python -m paper_2608_13499_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in EXPORTS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != OPSCALE_OK:
        lib = load()
        raise OpscaleError(status, lib.opscale_last_error().decode())


# ----------------------------------------------------------------- helpers --
def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return OPSCALE_BF16
    if t.dtype == torch.float32:
        return OPSCALE_F32
    raise OpscaleError(OPSCALE_ERR_UNSUPPORTED, f"dtype {t.dtype} (supported: bfloat16, float32)")


def _dev(*tensors):
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "tensors must be on the GPU")


def _stream(stream) -> int:
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def _contig(name, t):
    if not t.is_contiguous():
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, f"{name} must be contiguous")


# --------------------------------------------------------------- operators --
def _heads_view(name, t_, H, D):
    if t_.dim() != 3 or t_.shape[1] != H or t_.shape[2] != D or t_.stride(2) != 1 or t_.stride(1) != D:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, f"{name} must be [T, {H}, {D}] with contiguous heads")


def opscale_version() -> str:
    return load().opscale_version().decode()


def opscale_rmsnorm(x, w, y=None, eps: float = 1e-5, stream=None, timed: bool = False):
    """y = x / sqrt(mean(x^2) + eps) * w over the last dim of x [M, H]."""
    import torch
    lib = load()
    _dev(x, w, y)
    _contig("x", x)
    _contig("w", w)
    if y is None:
        y = torch.empty_like(x)
    _contig("y", y)
    H = x.shape[-1]
    M = x.numel() // H if H else 0
    t = Timing() if timed else None
    _check(lib.opscale_rmsnorm(_ptr(x), _ptr(w), _ptr(y), M, H, eps, _dt(x), _stream(stream),
                               ctypes.byref(t) if t else None))
    return (y, t) if timed else y


def opscale_set_tuning(knob: int, value: int):
    """Force (value >= 0) or release (-1) one of the library's path choices."""
    _check(load().opscale_set_tuning(knob, value))


def opscale_get_tuning(knob: int) -> int:
    return int(load().opscale_get_tuning(knob))


def opscale_linear_workspace_size(M: int, N: int, K: int, dtype=None) -> int:
    import torch
    dt = OPSCALE_F32 if dtype == torch.float32 else OPSCALE_BF16
    return int(load().opscale_linear_workspace_size(M, N, K, dt))


def _linear_shapes(x, W):
    K = x.shape[-1]
    if W.shape[1] != K:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, f"W is {tuple(W.shape)}, expected [N, {K}]")
    return x.numel() // K, W.shape[0], K


def _linear_workspace(x, W, workspace):
    """The workspace tensor to pass: given, allocated by torch (None), or none
    at all (False: the library then takes a path that needs none)."""
    import torch
    if workspace is False:
        return None
    if workspace is None:
        M, N, K = _linear_shapes(x, W)
        need = opscale_linear_workspace_size(M, N, K, x.dtype) if M else 0
        return torch.empty(need, dtype=torch.uint8, device=x.device) if need else None
    return workspace


def opscale_linear(x, W, bias=None, y=None, workspace=None, stream=None, timed: bool = False):
    """y[M, N] = x[M, K] W[N, K]^T (+ bias).  `workspace` (a uint8 GPU tensor)
    is allocated by torch when None; False passes none."""
    import torch
    lib = load()
    _dev(x, W, bias, y, workspace if workspace is not False else None)
    for n, t_ in (("x", x), ("W", W), ("bias", bias), ("y", y)):
        if t_ is not None:
            _contig(n, t_)
    M, N, K = _linear_shapes(x, W)
    if y is None:
        y = torch.empty(*x.shape[:-1], N, dtype=x.dtype, device=x.device)
    ws = _linear_workspace(x, W, workspace)
    t = Timing() if timed else None
    _check(lib.opscale_linear(_ptr(x), _ptr(W), _ptr(bias), _ptr(y), M, N, K, _dt(x), _ptr(ws),
                              0 if ws is None else ws.numel() * ws.element_size(), _stream(stream),
                              ctypes.byref(t) if t else None))
    return (y, t) if timed else y


def opscale_swiglu(gate_up, out=None, stream=None, timed: bool = False):
    """out[M, F] = silu(gate_up[:, :F]) * gate_up[:, F:]."""
    import torch
    lib = load()
    _dev(gate_up, out)
    _contig("gate_up", gate_up)
    F = gate_up.shape[-1] // 2
    M = gate_up.numel() // (2 * F)
    if out is None:
        out = torch.empty(*gate_up.shape[:-1], F, dtype=gate_up.dtype, device=gate_up.device)
    _contig("out", out)
    t = Timing() if timed else None
    _check(lib.opscale_swiglu(_ptr(gate_up), _ptr(out), M, F, _dt(gate_up), _stream(stream),
                              ctypes.byref(t) if t else None))
    return (out, t) if timed else out


def opscale_attn_prefill(q, k, v, cu_seqlens, max_seqlen: int, scale: float, causal: bool = True,
                         out=None, stream=None, timed: bool = False):
    """Ragged causal GQA attention.  q [T, Hq, D], k/v [T, Hkv, D]; the token
    dimension may be strided (views into a packed QKV tensor), heads and head
    dim must be contiguous.  cu_seqlens: int32 [B+1] on the GPU."""
    import torch
    lib = load()
    _dev(q, k, v, cu_seqlens, out)
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    for name, t_, H in (("q", q, Hq), ("k", k, Hkv), ("v", v, Hkv)):
        if t_.stride(2) != 1 or t_.stride(1) != D or t_.shape[0] != T:
            raise OpscaleError(OPSCALE_ERR_INVALID_ARG, f"{name} must be [T, H, D] with contiguous heads")
    if k.stride(0) != v.stride(0):
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "k and v must share a row stride")
    if cu_seqlens.dtype != torch.int32:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "cu_seqlens must be int32")
    if out is None:
        out = torch.empty(T, Hq, D, dtype=q.dtype, device=q.device)
    _contig("out", out)
    B = cu_seqlens.numel() - 1
    t = Timing() if timed else None
    _check(lib.opscale_attn_prefill(_ptr(q), _ptr(k), _ptr(v), q.stride(0), k.stride(0), _ptr(out),
                                    _ptr(cu_seqlens), B, T, max_seqlen, Hq, Hkv, D, scale, int(causal),
                                    _dt(q), _stream(stream), ctypes.byref(t) if t else None))
    return (out, t) if timed else out


def opscale_attn_decode_workspace_size(B: int, Hq: int, D: int, max_context_len: int) -> int:
    return int(load().opscale_attn_decode_workspace_size(B, Hq, D, max_context_len))


def opscale_attn_decode(q, k_cache, v_cache, block_table, context_lens, max_context_len: int,
                        scale: float, workspace=None, out=None, stream=None, timed: bool = False):
    """Decode attention over a paged cache [num_blocks, block_size, Hkv, D].
    q [B, Hq, D] may be strided in its first dimension (a view into the QKV
    output).  block_table int32 [B, max_blocks]; context_lens int32 [B].
    `workspace` (a uint8 GPU tensor) is allocated by torch when not given."""
    import torch
    lib = load()
    _dev(q, k_cache, v_cache, block_table, context_lens, workspace, out)
    for n, t_ in (("k_cache", k_cache), ("v_cache", v_cache), ("block_table", block_table),
                  ("context_lens", context_lens)):
        _contig(n, t_)
    B, Hq, D = q.shape
    _heads_view("q", q, Hq, D)
    num_blocks, bs, Hkv, _ = k_cache.shape
    need = opscale_attn_decode_workspace_size(B, Hq, D, max_context_len)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=q.dtype, device=q.device)
    _contig("out", out)
    t = Timing() if timed else None
    _check(lib.opscale_attn_decode(_ptr(q), q.stride(0), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                   _ptr(context_lens), _ptr(out), B, Hq, Hkv, D, bs, block_table.shape[1],
                                   num_blocks, max_context_len, scale, _dt(q), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream),
                                   ctypes.byref(t) if t else None))
    return (out, t) if timed else out


def opscale_attn_decode_noalloc(q, k_cache, v_cache, block_table, context_lens, max_context_len: int,
                                scale: float, out, stream=None):
    """opscale_attn_decode with the library's own scratch (no workspace, no
    allocation, no timing).  `out` [B, Hq, D] must be given."""
    lib = load()
    _dev(q, k_cache, v_cache, block_table, context_lens, out)
    for n, t_ in (("k_cache", k_cache), ("v_cache", v_cache), ("block_table", block_table),
                  ("context_lens", context_lens), ("out", out)):
        _contig(n, t_)
    B, Hq, D = q.shape
    _heads_view("q", q, Hq, D)
    num_blocks, bs, Hkv, _ = k_cache.shape
    _check(lib.opscale_attn_decode_noalloc(_ptr(q), q.stride(0), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                           _ptr(context_lens), _ptr(out), B, Hq, Hkv, D, bs, block_table.shape[1],
                                           num_blocks, max_context_len, scale, _dt(q), _stream(stream)))
    return out


def opscale_attn_decode_noalloc_max_bytes() -> int:
    return int(load().opscale_attn_decode_noalloc_max_bytes())


def opscale_rope(q, k, positions, theta: float, stream=None, timed: bool = False):
    """Rotary embedding of q [T, Hq, D] and k [T, Hkv, D] in place (rotate-half
    form); the token dimension may be strided (views into the QKV output).
    positions: int32 [T] on the GPU.  Returns (q, k)."""
    import torch
    lib = load()
    _dev(q, k, positions)
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    _heads_view("q", q, Hq, D)
    _heads_view("k", k, Hkv, D)
    if k.shape[0] != T or positions.dtype != torch.int32 or positions.numel() != T:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "k must have T rows and positions be int32 [T]")
    _contig("positions", positions)
    t = Timing() if timed else None
    _check(lib.opscale_rope(_ptr(q), _ptr(k), q.stride(0), k.stride(0), _ptr(positions), T, Hq, Hkv, D,
                            float(theta), _dt(q), _stream(stream), ctypes.byref(t) if t else None))
    return ((q, k), t) if timed else (q, k)


def opscale_reshape_and_cache(k, v, k_cache, v_cache, slot_mapping, stream=None, timed: bool = False):
    """Write k, v [T, Hkv, D] (token dimension may be strided) into the paged
    caches [num_blocks, block_size, Hkv, D] at the int32 slots; slots outside
    the cache are skipped."""
    import torch
    lib = load()
    _dev(k, v, k_cache, v_cache, slot_mapping)
    T, Hkv, D = k.shape
    _heads_view("k", k, Hkv, D)
    _heads_view("v", v, Hkv, D)
    if k.stride(0) != v.stride(0):
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "k and v must share a row stride")
    for n, t_ in (("k_cache", k_cache), ("v_cache", v_cache), ("slot_mapping", slot_mapping)):
        _contig(n, t_)
    if slot_mapping.dtype != torch.int32 or slot_mapping.numel() != T:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "slot_mapping must be int32 [T]")
    nb, bs = k_cache.shape[0], k_cache.shape[1]
    if tuple(k_cache.shape) != (nb, bs, Hkv, D) or tuple(v_cache.shape) != tuple(k_cache.shape):
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, f"caches must be [num_blocks, block_size, {Hkv}, {D}]")
    t = Timing() if timed else None
    _check(lib.opscale_reshape_and_cache(_ptr(k), _ptr(v), k.stride(0), _ptr(k_cache), _ptr(v_cache),
                                         _ptr(slot_mapping), T, Hkv, D, bs, nb, _dt(k), _stream(stream),
                                         ctypes.byref(t) if t else None))
    return t if timed else None


def opscale_add_rmsnorm(x, residual, w, y=None, eps: float = 1e-5, stream=None, timed: bool = False):
    """residual <- x + residual; y = rmsnorm(residual) * w.  Returns y."""
    import torch
    lib = load()
    _dev(x, residual, w, y)
    for n, t_ in (("x", x), ("residual", residual), ("w", w)):
        _contig(n, t_)
    if y is None:
        y = torch.empty_like(x)
    _contig("y", y)
    H = x.shape[-1]
    M = x.numel() // H if H else 0
    t = Timing() if timed else None
    _check(lib.opscale_add_rmsnorm(_ptr(x), _ptr(residual), _ptr(w), _ptr(y), M, H, eps, _dt(x), _stream(stream),
                                   ctypes.byref(t) if t else None))
    return (y, t) if timed else y


def opscale_op_profile(desc: OpDesc, warmup: int = 5, iters: int = 20, flush=None, stream=None) -> Profile:
    """Profile one operator call described by `desc` (see make_desc_*)."""
    lib = load()
    p = Profile()
    nbytes = 0 if flush is None else flush.numel() * flush.element_size()
    _check(lib.opscale_op_profile(ctypes.byref(desc), warmup, iters, _ptr(flush), nbytes,
                                  _stream(stream), ctypes.byref(p)))
    return p


# ------------------------------------------------------- mixture of experts --
def opscale_moe_topk(logits, topk: int, renormalize: bool = False, ids=None, weights=None, stream=None,
                     timed: bool = False):
    """Top-k routing of fp32 logits [T, E]: (ids int32 [T, topk], weights fp32 [T, topk])."""
    import torch
    _dev(logits)
    if logits.dtype != torch.float32 or logits.dim() != 2 or not logits.is_contiguous():
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "logits must be a contiguous float32 [T, E] tensor")
    T, E = logits.shape
    ids = torch.empty(T, topk, dtype=torch.int32, device=logits.device) if ids is None else ids
    weights = torch.empty(T, topk, dtype=torch.float32, device=logits.device) if weights is None else weights
    t = Timing() if timed else None
    _check(load().opscale_moe_topk(_ptr(logits), _ptr(ids), _ptr(weights), T, E, topk, int(renormalize),
                                   _stream(stream), ctypes.byref(t) if t else None))
    return (ids, weights, t) if timed else (ids, weights)


def opscale_fused_moe_workspace_size(T: int, H: int, F: int, E: int, topk: int) -> int:
    return int(load().opscale_fused_moe_workspace_size(T, H, F, E, topk))


def opscale_fused_moe(x, w1, w2, topk_ids, topk_weights, out=None, workspace=None, stream=None, timed: bool = False):
    """out[t] = sum_j w[t, j] * MLP_e(x[t]) over the routed experts; x [T, H] bf16,
    w1 [E, 2F, H], w2 [E, H, F]; topk_ids int32 / topk_weights fp32 [T, topk]."""
    import torch
    _dev(x, w1, w2, topk_ids, topk_weights)
    for name, t_ in (("x", x), ("w1", w1), ("w2", w2), ("topk_ids", topk_ids), ("topk_weights", topk_weights)):
        _contig(name, t_)
    T, H = x.shape
    E, F2, _ = w1.shape
    topk = topk_ids.shape[1]
    out = torch.empty_like(x) if out is None else out
    need = opscale_fused_moe_workspace_size(T, H, F2 // 2, E, topk)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    t = Timing() if timed else None
    _check(load().opscale_fused_moe(_ptr(x), _ptr(w1), _ptr(w2), _ptr(topk_ids), _ptr(topk_weights), _ptr(out), T,
                                    H, F2 // 2, E, topk, _dt(x), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _stream(stream),
                                    ctypes.byref(t) if t else None))
    return (out, t) if timed else out


def desc_fused_moe(x, w1, w2, topk_ids, topk_weights, out, workspace) -> OpDesc:
    d = OpDesc(op=OP_FUSED_MOE, dt=_dt(x))
    T, H = x.shape
    E, F2, _ = w1.shape
    d.u.fused_moe = _FusedMoeArgs(_ptr(x), _ptr(w1), _ptr(w2), _ptr(topk_ids), _ptr(topk_weights), _ptr(out), T, H,
                                  F2 // 2, E, topk_ids.shape[1], _ptr(workspace),
                                  workspace.numel() * workspace.element_size())
    return d


# ---------------------------------------------------------- spatial sharing --
def opscale_cu_layout():
    """(num_cus, num_xcds, interleaved) of the current device."""
    lib = load()
    n, x, i = c_i32(), c_i32(), c_i32()
    _check(lib.opscale_cu_layout(ctypes.byref(n), ctypes.byref(x), ctypes.byref(i)))
    return n.value, x.value, i.value


def opscale_cu_mask_build(num_cus: int, num_xcds: int, interleaved: int, first: int, count: int):
    """The CU mask (list of uint32 words) of balanced positions [first, first + count)."""
    lib = load()
    words = (num_cus + 31) // 32
    buf = (ctypes.c_uint32 * words)()
    _check(lib.opscale_cu_mask_build(num_cus, num_xcds, interleaved, first, count, buf, words))
    return list(buf)


def opscale_cu_stream_create(mask) -> int:
    """A CU-masked stream (an integer hipStream_t handle) for the uint32 words `mask`."""
    lib = load()
    buf = (ctypes.c_uint32 * len(mask))(*mask)
    h = c_vp()
    _check(lib.opscale_cu_stream_create(buf, len(mask), ctypes.byref(h)))
    return h.value


def opscale_cu_stream_destroy(stream: int):
    _check(load().opscale_cu_stream_destroy(stream))


def opscale_cu_stream_mask(stream: int, words: int):
    buf = (ctypes.c_uint32 * words)()
    _check(load().opscale_cu_stream_mask(stream, buf, words))
    return list(buf)


def opscale_cu_probe(out, spins: int = 4, stream=None):
    """Launch the placement probe: out is an int32 [n, 2] GPU tensor (XCD, HW_ID per workgroup)."""
    _dev(out)
    if out.dim() != 2 or out.shape[1] != 2 or not out.is_contiguous() or out.element_size() != 4:
        raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "out must be a contiguous 4-byte [n, 2] tensor")
    _check(load().opscale_cu_probe(_stream(stream), _ptr(out), out.shape[0], spins))
    return out


def opscale_probe_mfma(iters: int = 4096, reps: int = 5, stream=None) -> float:
    """Measured bf16 MFMA throughput of this GPU (TFLOP/s), blocking."""
    out = c_f64(0.0)
    _check(load().opscale_probe_mfma(int(iters), int(reps), _stream(stream), ctypes.byref(out)))
    return out.value


def opscale_probe_hbm(src, dst=None, reps: int = 5, stream=None) -> float:
    """Measured HBM streaming rate (GB/s), blocking: reads of src (a GPU
    tensor), or with dst (same byte size) a copy, counted as read + write."""
    _dev(src)
    nbytes = src.numel() * src.element_size()
    if dst is not None:
        _dev(dst)
        if dst.numel() * dst.element_size() != nbytes:
            raise OpscaleError(OPSCALE_ERR_INVALID_ARG, "dst must have the byte size of src")
    out = c_f64(0.0)
    _check(load().opscale_probe_hbm(_ptr(src), None if dst is None else _ptr(dst), nbytes, int(reps),
                                    _stream(stream), ctypes.byref(out)))
    return out.value


def opscale_corun_profile(desc_a: OpDesc, stream_a, desc_b: OpDesc, stream_b, warmup: int = 3,
                          iso_iters: int = 20, window_ms: float = 20.0, max_launches: int = 2048,
                          trace: bool = False):
    """Eq. 5 interference factors of two operators run at once on two streams.
    Returns a Corun (and, with trace=True, a dict of the raw launch times)."""
    lib = load()
    r = Corun()
    tr = None
    arrays = None
    if trace:
        arrays = {k: (c_f32 * n)() for k, n in (("a_start", max_launches), ("a_end", max_launches),
                                                ("b_start", max_launches), ("b_end", max_launches),
                                                ("a_iso", iso_iters), ("b_iso", iso_iters))}
        tr = _CorunTrace(**{k: ctypes.cast(v, _PF) for k, v in arrays.items()})
    _check(lib.opscale_corun_profile(ctypes.byref(desc_a), _stream(stream_a), ctypes.byref(desc_b),
                                     _stream(stream_b), warmup, iso_iters, window_ms, max_launches,
                                     ctypes.byref(tr) if tr is not None else None, ctypes.byref(r)))
    if not trace:
        return r
    n = {"a_start": r.n_a, "a_end": r.n_a, "b_start": r.n_b, "b_end": r.n_b, "a_iso": iso_iters,
         "b_iso": iso_iters}
    return r, {k: list(v)[:n[k]] for k, v in arrays.items()}


# descriptor builders (keep the tensors alive while the descriptor is used)
def desc_rmsnorm(x, w, y, eps=1e-5) -> OpDesc:
    d = OpDesc(op=OP_RMSNORM, dt=_dt(x))
    H = x.shape[-1]
    d.u.rmsnorm = _RmsnormArgs(_ptr(x), _ptr(w), _ptr(y), x.numel() // H, H, eps)
    return d


def desc_linear(x, W, y, bias=None, workspace=None) -> OpDesc:
    """`workspace` must stay alive while the descriptor is used (see
    opscale_linear for None / False)."""
    d = OpDesc(op=OP_LINEAR, dt=_dt(x))
    M, N, K = _linear_shapes(x, W)
    ws = _linear_workspace(x, W, workspace)
    d.u.linear = _LinearArgs(_ptr(x), _ptr(W), _ptr(bias), _ptr(y), M, N, K, _ptr(ws),
                             0 if ws is None else ws.numel() * ws.element_size())
    d._keep = ws
    return d


def desc_swiglu(gate_up, out) -> OpDesc:
    d = OpDesc(op=OP_SWIGLU, dt=_dt(gate_up))
    F = gate_up.shape[-1] // 2
    d.u.swiglu = _SwigluArgs(_ptr(gate_up), _ptr(out), gate_up.numel() // (2 * F), F)
    return d


def desc_attn_prefill(q, k, v, out, cu_seqlens, max_seqlen, scale, causal=True) -> OpDesc:
    d = OpDesc(op=OP_ATTN_PREFILL, dt=_dt(q))
    T, Hq, D = q.shape
    d.u.attn_prefill = _PrefillArgs(_ptr(q), _ptr(k), _ptr(v), q.stride(0), k.stride(0), _ptr(out),
                                    _ptr(cu_seqlens), cu_seqlens.numel() - 1, T, max_seqlen, Hq,
                                    k.shape[1], D, scale, int(causal))
    return d


def desc_attn_decode(q, k_cache, v_cache, block_table, context_lens, out, max_context_len, scale,
                     workspace) -> OpDesc:
    d = OpDesc(op=OP_ATTN_DECODE, dt=_dt(q))
    B, Hq, D = q.shape
    nb, bs, Hkv, _ = k_cache.shape
    _heads_view("q", q, Hq, D)
    d.u.attn_decode = _DecodeArgs(_ptr(q), q.stride(0), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                  _ptr(context_lens), _ptr(out), B, Hq, Hkv, D, bs, block_table.shape[1],
                                  nb, max_context_len, scale, _ptr(workspace),
                                  workspace.numel() * workspace.element_size())
    return d


def desc_rope(q, k, positions, theta) -> OpDesc:
    d = OpDesc(op=OP_ROPE, dt=_dt(q))
    T, Hq, D = q.shape
    _heads_view("q", q, Hq, D)
    _heads_view("k", k, k.shape[1], D)
    d.u.rope = _RopeArgs(_ptr(q), _ptr(k), q.stride(0), k.stride(0), _ptr(positions), T, Hq, k.shape[1], D,
                         float(theta))
    return d


def desc_reshape_and_cache(k, v, k_cache, v_cache, slot_mapping) -> OpDesc:
    d = OpDesc(op=OP_RESHAPE_AND_CACHE, dt=_dt(k))
    T, Hkv, D = k.shape
    nb, bs = k_cache.shape[0], k_cache.shape[1]
    d.u.reshape_and_cache = _CacheWriteArgs(_ptr(k), _ptr(v), k.stride(0), _ptr(k_cache), _ptr(v_cache),
                                            _ptr(slot_mapping), T, Hkv, D, bs, nb)
    return d


def desc_add_rmsnorm(x, residual, w, y, eps=1e-5) -> OpDesc:
    d = OpDesc(op=OP_ADD_RMSNORM, dt=_dt(x))
    H = x.shape[-1]
    d.u.add_rmsnorm = _AddRmsnormArgs(_ptr(x), _ptr(residual), _ptr(w), _ptr(y), x.numel() // H, H, eps)
    return d
