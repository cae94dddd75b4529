"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every symbol include/opscale.h declares, and rejects bad arguments with the
documented status codes before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "opscale.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(opscale_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    import paper_2608_13499_amd as ops
    return ops.load()


def test_header_declares_expected_entry_points():
    d = _declared()
    for name in ("opscale_rmsnorm", "opscale_linear", "opscale_swiglu", "opscale_attn_prefill",
                 "opscale_attn_decode", "opscale_attn_decode_workspace_size", "opscale_op_profile",
                 "opscale_version", "opscale_status_string", "opscale_last_error",
                 "opscale_rope", "opscale_reshape_and_cache", "opscale_add_rmsnorm",
                 "opscale_cu_layout", "opscale_cu_mask_build", "opscale_cu_stream_create",
                 "opscale_cu_stream_destroy", "opscale_cu_stream_mask", "opscale_cu_probe", "opscale_probe_mfma", "opscale_probe_hbm",
                 "opscale_corun_profile", "opscale_moe_topk", "opscale_fused_moe",
                 "opscale_fused_moe_workspace_size"):
        assert name in d


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    import paper_2608_13499_amd as ops
    assert set(_declared()) <= set(ops.EXPORTS)


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.opscale_version()
    assert lib.opscale_status_string(0) == b"ok"
    assert lib.opscale_status_string(3) == b"workspace too small"


P = ctypes.c_void_p
A16 = 1 << 20  # a 16-byte aligned fake address: never dereferenced, validation fails first


def _err(lib):
    return lib.opscale_last_error().decode()


def test_rmsnorm_validation(lib):
    assert lib.opscale_rmsnorm(None, None, None, 4, 4096, 1e-5, 1, None, None) == 1
    assert "null" in _err(lib)
    assert lib.opscale_rmsnorm(A16, A16, A16 * 2, 4, 4095, 1e-5, 1, None, None) == 1  # H*2 % 16
    assert lib.opscale_rmsnorm(A16 + 2, A16, A16 * 4, 4, 4096, 1e-5, 1, None, None) == 1  # misaligned
    assert lib.opscale_rmsnorm(A16, A16, A16 * 4, -1, 4096, 1e-5, 1, None, None) == 1
    assert lib.opscale_rmsnorm(A16, A16, A16 * 4, 4, 4096, -1.0, 1, None, None) == 1
    assert lib.opscale_rmsnorm(A16, A16, A16 * 4, 4, 4096, 1e-5, 7, None, None) == 1  # dtype
    assert lib.opscale_rmsnorm(A16, A16, A16 + 16, 4, 4096, 1e-5, 1, None, None) == 1  # partial overlap
    assert "overlap" in _err(lib)
    assert lib.opscale_rmsnorm(None, None, None, 0, 4096, 1e-5, 1, None, None) == 0  # empty: no-op


def test_linear_validation(lib):
    f = lib.opscale_linear
    assert f(A16, A16 * 2, None, A16 * 4, 8, 256, 100, 1, None, 0, None, None) == 1  # K*2 % 16
    assert f(A16, A16 * 2, None, A16 * 4, 8, 12, 64, 1, None, 0, None, None) == 1  # N*2 % 16
    assert f(A16, A16 * 2, None, A16, 8, 256, 64, 1, None, 0, None, None) == 1  # y aliases x
    assert f(A16, None, None, A16 * 4, 8, 256, 64, 1, None, 0, None, None) == 1
    assert f(A16, A16 * 2, A16 + 4, A16 * 4, 8, 256, 64, 1, None, 0, None, None) == 1  # bias align
    assert f(None, None, None, None, 0, 256, 64, 1, None, 0, None, None) == 0


G = 1 << 34  # fake addresses spaced far apart (never dereferenced)


def test_linear_workspace(lib):
    """The split partials live in a caller workspace whose size the query
    returns; too small a workspace is rejected before anything is enqueued."""
    size = lib.opscale_linear_workspace_size
    # 100 rows: the decode-batch kernel's 128-column tiles, 32 of them over
    # N = 4096, so K = 4096 (8 rounds of 8 slices) splits into
    # min(256 / 32, 8) = 8 ranges of fp32 [M, N] partials
    assert size(100, 4096, 4096, 1) == 8 * 100 * 4096 * 4
    # 128 rows: QKV's 48 tiles -> min(5, 8) = 5 ranges rounded to whole
    # rounds: 2 rounds each, 4 ranges; gate-up's 224 tiles fill the GPU unsplit
    assert size(128, 6144, 4096, 1) == 4 * 128 * 6144 * 4
    assert size(128, 28672, 4096, 1) == 0
    # 256 rows: the split-K tiles (128 x 256, 2 x 16 over N = 4096): 8 ranges
    assert size(256, 4096, 4096, 1) == 8 * 256 * 4096 * 4
    # the 8871-token gate-up projection: 35 x 112 tiles of 256 x 256 leave a
    # last round of 80 tiles, split into min(4, 256 // 80, 4096 // 512) = 3
    # K ranges of compact fp32 tiles
    assert size(8871, 28672, 4096, 1) == 3 * 80 * 256 * 256 * 4
    assert size(8, 4096, 4096, 1) == 0  # small-M kernel: reduces in LDS
    assert size(100, 4096, 4096, 0) == 0  # fp32 path
    assert size(0, 4096, 4096, 1) == 0
    f = lib.opscale_linear
    need = size(100, 4096, 4096, 1)
    x, W, y, ws = G, 2 * G, 3 * G, 4 * G
    assert f(x, W, None, y, 100, 4096, 4096, 1, ws, need - 1, None, None) == 3
    assert "workspace" in _err(lib)
    assert f(x, W, None, y, 100, 4096, 4096, 1, ws + 8, need, None, None) == 1  # misaligned
    assert f(x, W, None, y, 100, 4096, 4096, 1, y, need, None, None) == 1  # overlaps y
    assert "overlap" in _err(lib)


def test_tuning_hook(lib):
    TILE, SPLITK, NG = 0, 2, 4
    assert lib.opscale_set_tuning(99, 0) == 1 and lib.opscale_get_tuning(99) == -1
    assert lib.opscale_set_tuning(TILE, 4) == 1  # four tile forms: 0 .. 3
    assert lib.opscale_set_tuning(NG, 0) == 1  # 16 or 32 columns: 1, 2
    assert lib.opscale_get_tuning(SPLITK) == -1
    try:
        assert lib.opscale_set_tuning(SPLITK, 0) == 0 and lib.opscale_get_tuning(SPLITK) == 0
        assert lib.opscale_linear_workspace_size(100, 4096, 4096, 1) == 0  # no split planned
    finally:
        assert lib.opscale_set_tuning(SPLITK, -1) == 0
    assert lib.opscale_linear_workspace_size(100, 4096, 4096, 1) > 0


def test_swiglu_validation(lib):
    assert lib.opscale_swiglu(A16, A16, 8, 256, 1, None, None) == 1  # out overlaps input
    assert lib.opscale_swiglu(A16, A16 * 64, 8, 3, 0, None, None) == 1  # F*4 % 16
    assert lib.opscale_swiglu(None, None, 0, 256, 1, None, None) == 0


def test_prefill_validation(lib):
    f = lib.opscale_attn_prefill
    ok = dict(q=A16, k=A16, v=A16, qs=48 * 128, kvs=48 * 128, o=A16 * 8, cu=A16 * 16, B=2, T=100, ms=64,
              Hq=32, Hkv=8, D=128, scale=0.08, causal=1, dt=1)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["q"], a["k"], a["v"], a["qs"], a["kvs"], a["o"], a["cu"], a["B"], a["T"], a["ms"], a["Hq"],
                 a["Hkv"], a["D"], a["scale"], a["causal"], a["dt"], None, None)

    assert call(Hkv=5) == 1                # Hkv does not divide Hq
    assert call(D=96) == 2                 # unsupported head dim
    assert call(qs=100) == 1               # stride smaller than the heads
    assert call(ms=0) == 1
    assert call(cu=None) == 1
    assert call(scale=float("nan")) == 1
    assert call(scale=-0.5) == 1 and call(scale=0.0) == 1
    assert call(q=A16 + 8) == 1            # misaligned
    assert call(T=0) == 0 and call(B=0) == 0


def test_decode_validation_and_workspace(lib):
    f = lib.opscale_attn_decode
    need = lib.opscale_attn_decode_workspace_size(256, 32, 128, 8192)
    # balanced split-KV: one workgroup per 32-key tile of B x max_context_len
    # keys, at most 256 and 64 per sequence; the tile prefix sums (B + 1 int64), above 512
    # sequences each workgroup's first sequence (int32), each 256-byte aligned,
    # then (workgroups + B) x Hq partials of D + 2 floats
    def ws(B, Hq, D, mc):
        nwg = min(256, B * -(-mc // 32), 64 * B)
        up = lambda x: (x + 255) // 256 * 256
        return up(8 * (B + 1)) + (up(4 * nwg) if B > 512 else 0) + 4 * (nwg + B) * Hq * (D + 2)
    assert need == ws(256, 32, 128, 8192) == 2304 + 4 * (256 + 256) * 32 * 130
    assert lib.opscale_attn_decode_workspace_size(1, 32, 128, 2048) == 256 + 4 * (64 + 1) * 32 * 130
    assert lib.opscale_attn_decode_workspace_size(1, 32, 128, 8192) == 256 + 4 * (64 + 1) * 32 * 130
    for B, Hq, D, mc in [(1, 32, 128, 8192), (16, 32, 128, 2048), (64, 32, 128, 2048), (3, 8, 64, 33),
                         (1000, 64, 128, 1), (512, 8, 64, 100), (513, 8, 64, 100)]:
        assert lib.opscale_attn_decode_workspace_size(B, Hq, D, mc) == ws(B, Hq, D, mc)
    ok = dict(q=A16, qs=32 * 128, kc=A16, vc=A16, tab=A16, ctx=A16, o=A16 * 8, B=256, Hq=32, Hkv=8, D=128, bs=16,
              mb=512, nb=69424, mc=8192, scale=0.08, dt=1, ws=A16 * 32, wsb=need)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["q"], a["qs"], a["kc"], a["vc"], a["tab"], a["ctx"], a["o"], a["B"], a["Hq"], a["Hkv"], a["D"],
                 a["bs"], a["mb"], a["nb"], a["mc"], a["scale"], a["dt"], a["ws"], a["wsb"], None, None)

    assert call(wsb=need - 1) == 3
    assert call(ws=None) == 3
    assert call(bs=12) == 1                # not a power of two
    assert call(Hq=24, Hkv=8) == 2         # group of 3 unsupported on the bf16 path
    assert call(D=256) == 2
    assert call(tab=None) == 1
    assert call(mb=0) == 1
    assert call(qs=32 * 128 - 8) == 1      # stride smaller than the heads
    assert call(qs=48 * 128 + 4) == 1      # not a multiple of 16 bytes
    assert call(B=0) == 0


def test_rope_validation(lib):
    f = lib.opscale_rope
    ok = dict(q=A16, k=A16 * 2, qs=48 * 128, ks=48 * 128, pos=A16 * 4, T=100, Hq=32, Hkv=8, D=128, theta=5e5, dt=1)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["q"], a["k"], a["qs"], a["ks"], a["pos"], a["T"], a["Hq"], a["Hkv"], a["D"], a["theta"], a["dt"],
                 None, None)

    assert call(D=96) == 2
    assert call(theta=0.0) == 1 and call(theta=float("inf")) == 1
    assert call(qs=100) == 1               # smaller than the heads
    assert call(ks=8 * 128 + 4) == 1       # not a multiple of 16 bytes
    assert call(pos=None) == 1
    assert call(pos=A16 + 2) == 1          # misaligned positions
    assert call(q=A16 + 8) == 1
    assert call(T=0) == 0


def test_reshape_and_cache_validation(lib):
    f = lib.opscale_reshape_and_cache
    ok = dict(k=A16, v=A16 * 2, kvs=48 * 128, kc=A16 * 64, vc=A16 * 128, sl=A16 * 4, T=10, Hkv=8, D=128, bs=16,
              nb=1024, dt=1)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["k"], a["v"], a["kvs"], a["kc"], a["vc"], a["sl"], a["T"], a["Hkv"], a["D"], a["bs"], a["nb"],
                 a["dt"], None, None)

    assert call(D=3, Hkv=1) == 1            # a row is not a multiple of 16 bytes
    assert call(nb=1 << 27, bs=16) == 1     # slots do not fit in int32
    assert call(kvs=100) == 1
    assert call(sl=None) == 1
    assert call(kc=A16 + 16 * 1024) == 1    # k_cache overlaps k
    assert call(vc=A16 * 64 + 1024) == 1    # the caches overlap each other
    assert call(T=0) == 0


def test_add_rmsnorm_validation(lib):
    f = lib.opscale_add_rmsnorm
    assert f(A16, A16 * 4, A16 * 2, A16 * 8, 4, 16384, 1e-5, 1, None, None) == 2   # 32 KB rows
    assert f(A16, A16 + 32, A16 * 2, A16 * 8, 4, 4096, 1e-5, 1, None, None) == 1   # residual overlaps x
    assert f(A16, None, A16 * 2, A16 * 8, 4, 4096, 1e-5, 1, None, None) == 1
    assert f(A16, A16 * 4, A16 * 2, A16 * 4, 4, 4096, 1e-5, 1, None, None) == 1    # y is the residual


def test_profile_descriptor_layout_matches_header(tmp_path):
    """The ctypes mirror of opscale_op_desc / opscale_profile has the C layout
    (sizes and the offset of every union member's fields)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    import paper_2608_13499_amd as ops
    L = ops._lib
    members = {"rmsnorm": L._RmsnormArgs, "linear": L._LinearArgs, "swiglu": L._SwigluArgs,
               "attn_prefill": L._PrefillArgs, "attn_decode": L._DecodeArgs, "rope": L._RopeArgs,
               "reshape_and_cache": L._CacheWriteArgs, "add_rmsnorm": L._AddRmsnormArgs,
               "fused_moe": L._FusedMoeArgs}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "opscale.h"', "int main(void) {",
             'printf("desc_size %zu\\n", sizeof(opscale_op_desc));',
             'printf("desc_u %zu\\n", offsetof(opscale_op_desc, u));',
             'printf("profile %zu\\n", sizeof(opscale_profile));',
             'printf("corun %zu\\n", sizeof(opscale_corun));',
             'printf("corun_trace %zu\\n", sizeof(opscale_corun_trace));']
    for cname, cls in (("opscale_corun", L.Corun), ("opscale_corun_trace", L._CorunTrace)):
        for f, _ in cls._fields_:
            lines.append(f'printf("{cname}:{f} %zu\\n", offsetof({cname}, {f}));')
    for m, cls in members.items():
        for f, _ in cls._fields_:
            lines.append(f'printf("{m}.{f} %zu\\n", offsetof(opscale_op_desc, u.{m}.{f}) - '
                         f'offsetof(opscale_op_desc, u));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    r = subprocess.run(["gcc", "-I", HEADER.rsplit("/", 1)[0], "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__",
                        str(src), "-o", str(exe)], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("cannot compile against the HIP headers here: " + r.stderr[-200:])
    out = dict(line.rsplit(" ", 1) for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                               check=True).stdout.splitlines() if line)
    import ctypes
    assert int(out.pop("desc_size")) == ctypes.sizeof(L.OpDesc)
    assert int(out.pop("desc_u")) == L.OpDesc.u.offset
    assert int(out.pop("profile")) == ctypes.sizeof(L.Profile)
    assert int(out.pop("corun")) == ctypes.sizeof(L.Corun)
    assert int(out.pop("corun_trace")) == ctypes.sizeof(L._CorunTrace)
    for cname, cls in (("opscale_corun", L.Corun), ("opscale_corun_trace", L._CorunTrace)):
        for f, _ in cls._fields_:
            assert int(out.pop(f"{cname}:{f}")) == getattr(cls, f).offset, f"{cname}.{f}"
    for m, cls in members.items():
        for f, _ in cls._fields_:
            assert int(out[f"{m}.{f}"]) == getattr(cls, f).offset, f"{m}.{f}"


def test_probe_validation(lib):
    """The peak probes reject bad arguments before touching a device."""
    import ctypes
    out = ctypes.c_double(0.0)
    assert lib.opscale_probe_mfma(0, 5, None, ctypes.byref(out)) == 1          # iters < 1
    assert lib.opscale_probe_mfma(16, 0, None, ctypes.byref(out)) == 1         # reps < 1
    assert lib.opscale_probe_mfma(16, 5, None, None) == 1                      # no result pointer
    assert lib.opscale_probe_hbm(None, None, 1 << 20, 5, None, ctypes.byref(out)) == 1
    assert lib.opscale_probe_hbm(A16, None, 100, 5, None, ctypes.byref(out)) == 1      # not a multiple of 16
    assert lib.opscale_probe_hbm(A16 + 8, None, 1 << 20, 5, None, ctypes.byref(out)) == 1  # misaligned
    assert lib.opscale_probe_hbm(A16, None, 1 << 20, 0, None, ctypes.byref(out)) == 1  # reps < 1
    assert lib.opscale_probe_hbm(A16, A16 + 4096, 1 << 20, 5, None, ctypes.byref(out)) == 1  # dst overlaps src
    assert lib.opscale_probe_hbm(A16 + 4096, A16, 1 << 20, 5, None, ctypes.byref(out)) == 1  # src overlaps dst


def test_moe_validation(lib):
    f = lib.opscale_fused_moe
    need = lib.opscale_fused_moe_workspace_size(64, 128, 256, 8, 2)
    assert need > 64 * 2 * (2 * 256 + 256 + 128) * 2
    ok = dict(x=A16, w1=A16 * 2, w2=A16 * 4, ids=A16 * 6, wts=A16 * 7, out=A16 * 8, T=64, H=128, F=256, E=8, k=2,
              dt=1, ws=A16 * 16, wsb=need)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["x"], a["w1"], a["w2"], a["ids"], a["wts"], a["out"], a["T"], a["H"], a["F"], a["E"], a["k"],
                 a["dt"], a["ws"], a["wsb"], None, None)

    assert call(dt=0) == 2                      # fp32: bf16 only
    assert call(H=100) == 1 and call(F=4) == 1  # multiples of 8
    assert call(E=0) == 1 and call(E=1025) == 1
    assert call(k=0) == 1 and call(k=65) == 1
    assert call(wsb=need - 1) == 3
    assert call(x=A16 + 4) == 1                 # misaligned
    assert call(ids=A16 * 6 + 2) == 1
    assert call(out=A16 + 64) == 1              # out overlaps x
    assert call(T=1 << 24) == 2                 # T*H beyond the 32-bit offsets
    assert call(T=0) == 0
    t = lib.opscale_moe_topk
    assert t(A16, A16 * 2, A16 * 3, 10, 8, 9, 1, None, None) == 1   # topk > E
    assert t(A16, A16 * 2, A16 * 3, 10, 64, 17, 1, None, None) == 1  # topk > 16
    assert t(A16, A16 * 2, A16 * 3, 10, 2000, 2, 1, None, None) == 1
    assert t(None, None, None, 0, 8, 2, 1, None, None) == 0
