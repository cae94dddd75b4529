// C ABI of libopscale: argument validation, dispatch to the gfx950 kernels,
// kernel-only timing with device events and the per-operator profile.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "launch.h"
#include "opscale.h"
#include "status.h"

namespace opscale {

thread_local std::string g_last_error;

opscale_status fail(opscale_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

opscale_status hip_fail(hipError_t e, const char* what) {
  return fail(OPSCALE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// The tuning overrides (opscale_set_tuning); -1 everywhere means automatic.
namespace {
std::atomic<int32_t> g_tuning[OPSCALE_TUNE_COUNT] = {-1, -1, -1, -1, -1, -1, -1, -1};
}  // namespace

int32_t tuning(opscale_tune knob) {
  return (unsigned)knob < (unsigned)OPSCALE_TUNE_COUNT ? g_tuning[knob].load(std::memory_order_relaxed) : -1;
}

opscale_status set_tuning(opscale_tune knob, int32_t value) {
  if ((unsigned)knob >= (unsigned)OPSCALE_TUNE_COUNT)
    return fail(OPSCALE_ERR_INVALID_ARG, "set_tuning: unknown knob %d", (int)knob);
  int32_t hi = 1;
  if (knob == OPSCALE_TUNE_GEMM_TILE) hi = 3;
  if (knob == OPSCALE_TUNE_SKINNY_NG) hi = 2;
  const int32_t lo = knob == OPSCALE_TUNE_SKINNY_NG ? 1 : 0;
  if (value != -1 && (value < lo || value > hi))
    return fail(OPSCALE_ERR_INVALID_ARG, "set_tuning: value %d out of range for knob %d", (int)value, (int)knob);
  g_tuning[knob].store(value, std::memory_order_relaxed);
  return OPSCALE_OK;
}

}  // namespace opscale

namespace {

using opscale::fail;
using opscale::hip_fail;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int esize(opscale_dtype dt) { return dt == OPSCALE_BF16 ? 2 : 4; }

bool dtype_ok(opscale_dtype dt) { return dt == OPSCALE_F32 || dt == OPSCALE_BF16; }

// [a, a+na) and [b, b+nb) overlap?
bool overlap(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

constexpr int64_t kMaxDim = (int64_t)1 << 31;

// Events used to time one call on this host thread (created on first use).
struct ThreadEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  hipError_t init() {
    if (start) return hipSuccess;
    hipError_t e = hipEventCreate(&start);
    if (e != hipSuccess) return e;
    e = hipEventCreate(&stop);
    if (e != hipSuccess) {
      (void)hipEventDestroy(start);
      start = nullptr;
    }
    return e;
  }
};
thread_local ThreadEvents g_events;

// Runs `launch` on `s`, bracketed by events when `t` is non-null.
template <class F>
opscale_status run_timed(hipStream_t s, opscale_timing* t, const char* what, F&& launch) {
  if (t) {
    hipError_t e = g_events.init();
    if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    e = hipEventRecord(g_events.start, s);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  hipError_t e = launch();
  if (e != hipSuccess) return hip_fail(e, what);
  if (t) {
    e = hipEventRecord(g_events.stop, s);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    e = hipEventSynchronize(g_events.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, g_events.start, g_events.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    t->elapsed_us = ms * 1000.f;
  }
  return OPSCALE_OK;
}

void zero_timing(opscale_timing* t) {
  if (t) *t = opscale_timing{0.f, 0.0, 0.0};
}

// ------------------------------------------------------ algorithmic work ----
struct Work {
  double flops, bytes;
  int64_t weight, transient, io;
};

Work work_rmsnorm(int64_t M, int64_t H, int s) {
  return {4.0 * M * H, (double)s * (2.0 * M * H + H), s * H, s * 2 * M * H, s * M * H};
}
Work work_linear(int64_t M, int64_t N, int64_t K, int s, bool bias) {
  const double by = (double)s * ((double)M * K + (double)N * K + (double)M * N) + (bias ? (double)s * N : 0.0);
  return {2.0 * M * N * K, by, s * (N * K + (bias ? N : 0)), s * (M * K + M * N), s * M * N};
}
Work work_swiglu(int64_t M, int64_t F, int s) {
  return {6.0 * M * F, 3.0 * s * M * F, 0, 3 * s * M * F, s * M * F};
}
Work work_prefill(const std::vector<int32_t>& cu, int64_t Hq, int64_t Hkv, int64_t D, int s, bool causal) {
  double pairs = 0;
  for (size_t b = 0; b + 1 < cu.size(); ++b) {
    const double L = (double)(cu[b + 1] - cu[b]);
    pairs += causal ? L * (L + 1) / 2 : L * L;
  }
  const int64_t T = cu.empty() ? 0 : cu.back();
  const int64_t tb = (int64_t)s * (2 * T * Hq * D + 2 * T * Hkv * D);
  return {4.0 * D * Hq * pairs, (double)tb, 0, tb, (int64_t)s * T * Hq * D};
}
Work work_decode(const std::vector<int32_t>& ctx, int64_t Hq, int64_t Hkv, int64_t D, int s, int64_t bs,
                 int64_t max_blocks) {
  double N = 0, nb = 0;
  const int64_t B = (int64_t)ctx.size();
  for (int32_t c : ctx) {
    const int64_t n = std::min<int64_t>(std::max<int32_t>(c, 0), max_blocks * bs);
    N += n;
    nb += (double)((n + bs - 1) / bs);
  }
  const double by = s * (2.0 * Hkv * D * N + 2.0 * B * Hq * D) + 4.0 * (nb + B);
  return {4.0 * D * Hq * N, by, 0, (int64_t)by, s * B * Hq * D};
}

// weight: parameters read; transient: activations / cache touched; io: the
// payload handed to the next operator.
Work work_rope(int64_t T, int64_t Hq, int64_t Hkv, int64_t D, int s) {
  const int64_t qk = (int64_t)s * T * (Hq + Hkv) * D;
  return {3.0 * T * (Hq + Hkv) * D, 2.0 * qk + 4.0 * T, 0, qk, qk};
}
Work work_cache_write(int64_t T, int64_t Hkv, int64_t D, int s) {
  const int64_t kv = 2 * (int64_t)s * T * Hkv * D;
  return {0.0, 2.0 * kv + 4.0 * T, 0, kv, 0};
}
Work work_add_rmsnorm(int64_t M, int64_t H, int s) {
  return {5.0 * M * H, (double)s * (4.0 * M * H + H), s * H, s * 4 * M * H, s * 2 * M * H};
}

// MoE: each valid (token, slot) pair does the two expert GEMMs (2 H 2F + 2 F H
// flops, 6 H F) and the SwiGLU (6 F); x and out are read / written once and
// the weights of every expert that receives a token are read once.
Work work_fused_moe(const std::vector<int32_t>& ids, int64_t T, int64_t H, int64_t F, int64_t E, int s) {
  std::vector<char> used((size_t)E, 0);
  double pairs = 0;
  for (int32_t e : ids)
    if (e >= 0 && e < E) {
      used[(size_t)e] = 1;
      pairs += 1;
    }
  int64_t experts = 0;
  for (char u : used) experts += u;
  const int64_t weight = (int64_t)s * experts * 3 * H * F;
  const double by = (double)weight + 2.0 * s * T * H + 8.0 * (double)ids.size();
  return {pairs * (6.0 * H * F + 6.0 * F), by, weight, (int64_t)s * T * H + 8 * (int64_t)ids.size(),
          (int64_t)s * T * H};
}

opscale_status copy_ints(std::vector<int32_t>& dst, const int32_t* src, int64_t n, hipStream_t s) {
  dst.resize((size_t)n);
  if (n == 0) return OPSCALE_OK;
  hipError_t e = hipMemcpyAsync(dst.data(), src, (size_t)n * 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return e == hipSuccess ? OPSCALE_OK : hip_fail(e, "hipMemcpyAsync(lengths)");
}

// ------------------------------------------------------------ validation ----
opscale_status check_rmsnorm(const void* x, const void* w, void* y, int64_t M, int64_t H,
                             float eps, opscale_dtype dt) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: unknown dtype %d", (int)dt);
  if (M < 0 || H <= 0 || M >= kMaxDim || H > (1 << 24))
    return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: bad sizes M=%lld H=%lld", (long long)M, (long long)H);
  if ((H * esize(dt)) % 16)
    return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: H*sizeof(dt)=%lld is not a multiple of 16",
                (long long)(H * esize(dt)));
  if (!(eps >= 0.f) || std::isinf(eps)) return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: eps must be finite and >= 0");
  if (M == 0) return OPSCALE_OK;
  if (!x || !w || !y) return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: null pointer");
  if (!aligned16(x) || !aligned16(w) || !aligned16(y))
    return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: pointers must be 16-byte aligned");
  const int64_t nb = M * H * esize(dt);
  if (x != y && overlap(x, nb, y, nb))
    return fail(OPSCALE_ERR_INVALID_ARG, "rmsnorm: y partially overlaps x (only y == x is allowed)");
  return OPSCALE_OK;
}

opscale_status check_linear(const void* x, const void* W, const void* bias, void* y, int64_t M,
                            int64_t N, int64_t K, opscale_dtype dt, const void* ws, size_t ws_bytes,
                            opscale::LinearPlan* plan) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "linear: unknown dtype %d", (int)dt);
  if (M < 0 || N <= 0 || K <= 0 || M >= kMaxDim || N >= kMaxDim || K > (1 << 20))
    return fail(OPSCALE_ERR_INVALID_ARG, "linear: bad sizes M=%lld N=%lld K=%lld", (long long)M,
                (long long)N, (long long)K);
  const int s = esize(dt);
  if ((K * s) % 16 || (N * s) % 16)
    return fail(OPSCALE_ERR_INVALID_ARG, "linear: K and N times sizeof(dt) must be multiples of 16 (K=%lld N=%lld)",
                (long long)K, (long long)N);
  if (M == 0) return OPSCALE_OK;
  if (!x || !W || !y) return fail(OPSCALE_ERR_INVALID_ARG, "linear: null pointer");
  if (!aligned16(x) || !aligned16(W) || !aligned16(y) || (bias && !aligned16(bias)))
    return fail(OPSCALE_ERR_INVALID_ARG, "linear: pointers must be 16-byte aligned");
  if (overlap(y, M * N * s, x, M * K * s) || overlap(y, M * N * s, W, N * K * s))
    return fail(OPSCALE_ERR_INVALID_ARG, "linear: y must not overlap x or W");
  // no workspace: a path that needs none; a workspace: the path it allows,
  // which must then fit
  *plan = opscale::plan_linear(M, N, K, dt == OPSCALE_BF16, ws != nullptr);
  if (plan->ws_bytes > 0) {
    if (ws_bytes < plan->ws_bytes)
      return fail(OPSCALE_ERR_WORKSPACE, "linear: workspace of %zu bytes, %zu needed", ws_bytes, plan->ws_bytes);
    if (!aligned16(ws)) return fail(OPSCALE_ERR_INVALID_ARG, "linear: workspace must be 16-byte aligned");
    if (overlap(ws, (int64_t)plan->ws_bytes, y, M * N * s) || overlap(ws, (int64_t)plan->ws_bytes, x, M * K * s) ||
        overlap(ws, (int64_t)plan->ws_bytes, W, N * K * s))
      return fail(OPSCALE_ERR_INVALID_ARG, "linear: workspace overlaps x, W or y");
  }
  return OPSCALE_OK;
}

opscale_status check_swiglu(const void* gu, void* out, int64_t M, int64_t F, opscale_dtype dt) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: unknown dtype %d", (int)dt);
  if (M < 0 || F <= 0 || M >= kMaxDim || F >= kMaxDim)
    return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: bad sizes M=%lld F=%lld", (long long)M, (long long)F);
  const int s = esize(dt);
  if ((F * s) % 16)
    return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: F*sizeof(dt)=%lld is not a multiple of 16", (long long)(F * s));
  if (M == 0) return OPSCALE_OK;
  if (!gu || !out) return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: null pointer");
  if (!aligned16(gu) || !aligned16(out)) return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: pointers must be 16-byte aligned");
  if (overlap(gu, M * 2 * F * s, out, M * F * s))
    return fail(OPSCALE_ERR_INVALID_ARG, "swiglu: out must not overlap gate_up");
  return OPSCALE_OK;
}

opscale_status check_prefill(const void* q, const void* k, const void* v, int64_t qs, int64_t kvs,
                             void* o, const int32_t* cu, int32_t B, int64_t T, int32_t max_seqlen,
                             int32_t Hq, int32_t Hkv, int32_t D, float scale, opscale_dtype dt) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: unknown dtype %d", (int)dt);
  if (B < 0 || T < 0 || T >= kMaxDim || Hq <= 0 || Hkv <= 0)
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: bad sizes B=%d T=%lld Hq=%d Hkv=%d", B, (long long)T, Hq, Hkv);
  if (Hq % Hkv) return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: Hkv=%d does not divide Hq=%d", Hkv, Hq);
  if (D != 64 && D != 128) return fail(OPSCALE_ERR_UNSUPPORTED, "attn_prefill: head_dim %d (supported: 64, 128)", D);
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: scale must be finite and > 0");
  if (B == 0 || T == 0) return OPSCALE_OK;
  if (max_seqlen < 1) return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: max_seqlen must be >= 1");
  const int vec = 16 / esize(dt);
  if (qs < (int64_t)Hq * D || kvs < (int64_t)Hkv * D || qs % vec || kvs % vec || qs > (1 << 24) || kvs > (1 << 24))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: row strides q=%lld kv=%lld must cover the heads, be multiples of %d and <= 2^24",
                (long long)qs, (long long)kvs, vec);
  if (!q || !k || !v || !o || !cu) return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: null pointer");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || (reinterpret_cast<uintptr_t>(cu) & 3))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_prefill: q, k, v, o must be 16-byte aligned, cu_seqlens 4-byte");
  if ((int64_t)B * Hkv * Hq >= kMaxDim) return fail(OPSCALE_ERR_UNSUPPORTED, "attn_prefill: batch too large");
  return OPSCALE_OK;
}

opscale_status check_decode(const void* q, int64_t qs, const void* kc, const void* vc, const int32_t* table,
                            const int32_t* ctx, void* o, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                            int32_t bs, int32_t max_blocks, int64_t num_blocks, int32_t max_ctx,
                            float scale, opscale_dtype dt, void* ws, size_t ws_bytes) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: unknown dtype %d", (int)dt);
  if (B < 0 || Hq <= 0 || Hkv <= 0 || B > 65535 || Hq > 65535)
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: bad sizes B=%d Hq=%d Hkv=%d", B, Hq, Hkv);
  if (Hq % Hkv) return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: Hkv=%d does not divide Hq=%d", Hkv, Hq);
  if (D != 64 && D != 128) return fail(OPSCALE_ERR_UNSUPPORTED, "attn_decode: head_dim %d (supported: 64, 128)", D);
  const int G = Hq / Hkv;
  if (dt == OPSCALE_BF16 && G != 1 && G != 2 && G != 4 && G != 8)
    return fail(OPSCALE_ERR_UNSUPPORTED, "attn_decode: bf16 supports Hq/Hkv in {1, 2, 4, 8}, got %d", G);
  if (bs < 1 || bs > 1024 || (bs & (bs - 1)))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: block_size %d must be a power of two in [1, 1024]", bs);
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: scale must be finite and > 0");
  if (B == 0) return OPSCALE_OK;
  if (max_blocks < 1 || (int64_t)max_blocks * bs >= kMaxDim || num_blocks < 1 || max_ctx < 1)
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: max_blocks_per_seq=%d num_blocks=%lld max_context_len=%d",
                max_blocks, (long long)num_blocks, max_ctx);
  if (qs < (int64_t)Hq * D || qs % (16 / esize(dt)) || qs > (1 << 24))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: q_row_stride=%lld must cover the heads, be a multiple of 16 bytes and <= 2^24",
                (long long)qs);
  if (!q || !kc || !vc || !table || !ctx || !o) return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: null pointer");
  if (!aligned16(q) || !aligned16(kc) || !aligned16(vc) || !aligned16(o) ||
      (reinterpret_cast<uintptr_t>(table) & 3) || (reinterpret_cast<uintptr_t>(ctx) & 3))
    return fail(OPSCALE_ERR_INVALID_ARG, "attn_decode: tensors must be 16-byte aligned, indices 4-byte");
  const size_t need = opscale::decode_workspace_bytes(B, Hq, D, max_ctx);
  if (dt == OPSCALE_BF16 && (!ws || ws_bytes < need || !aligned16(ws)))
    return fail(OPSCALE_ERR_WORKSPACE, "attn_decode: workspace of %zu bytes (16-byte aligned) needed, got %zu",
                need, ws ? ws_bytes : (size_t)0);
  return OPSCALE_OK;
}

opscale_status check_rope(void* q, void* k, int64_t qs, int64_t ks, const int32_t* pos, int64_t T, int32_t Hq,
                          int32_t Hkv, int32_t D, double theta, opscale_dtype dt) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "rope: unknown dtype %d", (int)dt);
  if (T < 0 || T >= kMaxDim || Hq <= 0 || Hkv <= 0 || Hq > 65535 || Hkv > 65535)
    return fail(OPSCALE_ERR_INVALID_ARG, "rope: bad sizes T=%lld Hq=%d Hkv=%d", (long long)T, Hq, Hkv);
  if (D != 64 && D != 128) return fail(OPSCALE_ERR_UNSUPPORTED, "rope: head_dim %d (supported: 64, 128)", D);
  if (!(theta > 0.0) || !std::isfinite(theta)) return fail(OPSCALE_ERR_INVALID_ARG, "rope: theta must be finite and > 0");
  if (T == 0) return OPSCALE_OK;
  const int vec = 16 / esize(dt);
  if (qs < (int64_t)Hq * D || ks < (int64_t)Hkv * D || qs % vec || ks % vec)
    return fail(OPSCALE_ERR_INVALID_ARG, "rope: row strides q=%lld k=%lld must cover the heads and be multiples of %d",
                (long long)qs, (long long)ks, vec);
  if (!q || !k || !pos) return fail(OPSCALE_ERR_INVALID_ARG, "rope: null pointer");
  if (!aligned16(q) || !aligned16(k) || (reinterpret_cast<uintptr_t>(pos) & 3))
    return fail(OPSCALE_ERR_INVALID_ARG, "rope: q, k must be 16-byte aligned, positions 4-byte");
  return OPSCALE_OK;
}

opscale_status check_cache_write(const void* k, const void* v, int64_t kvs, void* kc, void* vc, const int32_t* slots,
                                 int64_t T, int32_t Hkv, int32_t D, int32_t bs, int64_t nb, opscale_dtype dt) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: unknown dtype %d", (int)dt);
  if (T < 0 || T >= kMaxDim || Hkv <= 0 || D <= 0 || (int64_t)Hkv * D > (1 << 20))
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: bad sizes T=%lld Hkv=%d D=%d", (long long)T, Hkv, D);
  const int s = esize(dt);
  if (((int64_t)Hkv * D * s) % 16)
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: a row (Hkv*D*sizeof(dt)) must be a multiple of 16 bytes");
  if (bs < 1 || nb < 1 || nb * bs >= ((int64_t)1 << 31))
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: block_size=%d num_blocks=%lld", bs, (long long)nb);
  if (T == 0) return OPSCALE_OK;
  if (kvs < (int64_t)Hkv * D || (kvs * s) % 16)
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: kv_row_stride=%lld must cover the heads and be a multiple of 16 bytes",
                (long long)kvs);
  if (!k || !v || !kc || !vc || !slots) return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: null pointer");
  if (!aligned16(k) || !aligned16(v) || !aligned16(kc) || !aligned16(vc) || (reinterpret_cast<uintptr_t>(slots) & 3))
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: tensors must be 16-byte aligned, slots 4-byte");
  const int64_t cache_bytes = nb * bs * Hkv * D * s, in_bytes = ((T - 1) * kvs + (int64_t)Hkv * D) * s;
  if (overlap(kc, cache_bytes, k, in_bytes) || overlap(kc, cache_bytes, v, in_bytes) ||
      overlap(vc, cache_bytes, k, in_bytes) || overlap(vc, cache_bytes, v, in_bytes) ||
      overlap(kc, cache_bytes, vc, cache_bytes))
    return fail(OPSCALE_ERR_INVALID_ARG, "reshape_and_cache: the caches must not overlap k, v or each other");
  return OPSCALE_OK;
}

opscale_status check_add_rmsnorm(const void* x, void* res, const void* w, void* y, int64_t M, int64_t H, float eps,
                                 opscale_dtype dt) {
  opscale_status st = check_rmsnorm(x, w, y, M, H, eps, dt);
  if (st != OPSCALE_OK || M == 0) return st;
  if (H * esize(dt) > 16384)
    return fail(OPSCALE_ERR_UNSUPPORTED, "add_rmsnorm: rows of up to 16 KB (H*sizeof(dt)), got %lld bytes",
                (long long)(H * esize(dt)));
  if (!res) return fail(OPSCALE_ERR_INVALID_ARG, "add_rmsnorm: null residual");
  if (!aligned16(res)) return fail(OPSCALE_ERR_INVALID_ARG, "add_rmsnorm: residual must be 16-byte aligned");
  const int64_t nb = M * H * esize(dt);
  if (overlap(res, nb, x, nb) || overlap(res, nb, y, nb) || overlap(res, nb, w, H * esize(dt)))
    return fail(OPSCALE_ERR_INVALID_ARG, "add_rmsnorm: residual must not overlap x, y or w");
  return OPSCALE_OK;
}

opscale_status check_moe_topk(const float* logits, int32_t* ids, float* wts, int64_t T, int32_t E, int32_t k) {
  if (T < 0 || T >= kMaxDim) return fail(OPSCALE_ERR_INVALID_ARG, "moe_topk: bad T=%lld", (long long)T);
  if (E < 1 || E > opscale::moe_max_experts())
    return fail(OPSCALE_ERR_INVALID_ARG, "moe_topk: E=%d outside [1, %d]", E, opscale::moe_max_experts());
  if (k < 1 || k > std::min<int32_t>(E, 16))
    return fail(OPSCALE_ERR_INVALID_ARG, "moe_topk: topk=%d outside [1, min(E, 16)]", k);
  if (T == 0) return OPSCALE_OK;
  if (!logits || !ids || !wts) return fail(OPSCALE_ERR_INVALID_ARG, "moe_topk: null pointer");
  if ((reinterpret_cast<uintptr_t>(logits) | reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(wts)) & 3)
    return fail(OPSCALE_ERR_INVALID_ARG, "moe_topk: pointers must be 4-byte aligned");
  return OPSCALE_OK;
}

opscale_status check_fused_moe(const void* x, const void* w1, const void* w2, const int32_t* ids, const float* wts,
                               void* out, int64_t T, int32_t H, int32_t F, int32_t E, int32_t k, opscale_dtype dt,
                               void* ws, size_t ws_bytes) {
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: unknown dtype %d", (int)dt);
  if (dt != OPSCALE_BF16) return fail(OPSCALE_ERR_UNSUPPORTED, "fused_moe: bf16 only");
  if (T < 0 || H < 8 || F < 8 || H % 8 || F % 8)
    return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: bad sizes T=%lld H=%d F=%d (H, F multiples of 8)",
                (long long)T, H, F);
  if (E < 1 || E > opscale::moe_max_experts())
    return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: E=%d outside [1, %d]", E, opscale::moe_max_experts());
  if (k < 1 || k > 64) return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: topk=%d outside [1, 64]", k);
  if (T * H >= (1ll << 30) || T * k * 2ll * F >= (1ll << 30))
    return fail(OPSCALE_ERR_UNSUPPORTED, "fused_moe: T*H and T*topk*2F must stay below 2^30");
  if (T == 0) return OPSCALE_OK;
  if (!x || !w1 || !w2 || !ids || !wts || !out || !ws) return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: null pointer");
  if (!aligned16(x) || !aligned16(w1) || !aligned16(w2) || !aligned16(out) || !aligned16(ws))
    return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: x, w1, w2, out and workspace must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(wts)) & 3)
    return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: topk_ids and topk_weights must be 4-byte aligned");
  if (overlap(out, T * H * 2, x, T * H * 2))
    return fail(OPSCALE_ERR_INVALID_ARG, "fused_moe: out must not overlap x");
  const size_t need = opscale::moe_workspace_bytes(T, H, F, E, k);
  if (ws_bytes < need)
    return fail(OPSCALE_ERR_WORKSPACE, "fused_moe: workspace of %zu bytes, %zu needed", ws_bytes, need);
  return OPSCALE_OK;
}

// Median with linear interpolation between the two middle values (the
// percentile rule of opscale_op_profile); 0 for an empty list.
float median_of(std::vector<float> v) {
  if (v.empty()) return 0.f;
  std::sort(v.begin(), v.end());
  const double pos = 0.5 * (double)(v.size() - 1);
  const size_t lo = (size_t)std::floor(pos), hi = (size_t)std::ceil(pos);
  return (float)(v[lo] + (v[hi] - v[lo]) * (pos - (double)lo));
}

// Owns a set of timing events.
struct EventPool {
  std::vector<hipEvent_t> ev;
  hipError_t make(size_t n) {
    ev.assign(n, nullptr);
    for (auto& e : ev) {
      const hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) return r;
    }
    return hipSuccess;
  }
  ~EventPool() {
    for (auto e : ev)
      if (e) (void)hipEventDestroy(e);
  }
};

// Per-launch times (us) of `n` back-to-back launches on s, each between two events.
opscale_status time_loop(const std::function<hipError_t()>& launch, hipStream_t s, int n, std::vector<float>* us) {
  EventPool pool;
  hipError_t e = pool.make((size_t)n + 1);
  if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
  if ((e = hipEventRecord(pool.ev[0], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  for (int i = 0; i < n; ++i) {
    if ((e = launch()) != hipSuccess) return hip_fail(e, "corun launch");
    if ((e = hipEventRecord(pool.ev[(size_t)i + 1], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  if ((e = hipEventSynchronize(pool.ev[(size_t)n])) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  us->resize((size_t)n);
  for (int i = 0; i < n; ++i) {
    float ms = 0.f;
    if ((e = hipEventElapsedTime(&ms, pool.ev[(size_t)i], pool.ev[(size_t)i + 1])) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
    (*us)[(size_t)i] = ms * 1000.f;
  }
  return OPSCALE_OK;
}

// ----------------------------------------- allocation-free decode scratch ---
// The scratch of opscale_attn_decode_noalloc: a file-scope device array.
// Each GPU the library runs on holds its own copy, at its own address, until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory, so its device address is looked up once per device (with
// that device current) and only that address is ever passed to a kernel.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

opscale_status static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(OPSCALE_ERR_UNSUPPORTED, "attn_decode_noalloc: device %d beyond the %d supported", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(OPSCALE_ERR_HIP, "hipGetSymbolAddress(scratch) returned no address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return OPSCALE_OK;
}

}  // namespace

extern "C" {

const char* opscale_version(void) { return "opscale 0.1.0 gfx950"; }

const char* opscale_status_string(opscale_status s) {
  switch (s) {
    case OPSCALE_OK: return "ok";
    case OPSCALE_ERR_INVALID_ARG: return "invalid argument";
    case OPSCALE_ERR_UNSUPPORTED: return "unsupported";
    case OPSCALE_ERR_WORKSPACE: return "workspace too small";
    case OPSCALE_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* opscale_last_error(void) { return opscale::g_last_error.c_str(); }

opscale_status opscale_rmsnorm(const void* x, const void* w, void* y, int64_t M, int64_t H, float eps,
                               opscale_dtype dt, hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_rmsnorm(x, w, y, M, H, eps, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (M == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "rmsnorm launch", [&] {
    return opscale::launch_rmsnorm(x, w, y, M, H, eps, dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_rmsnorm(M, H, esize(dt));
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_set_tuning(opscale_tune knob, int32_t value) { return opscale::set_tuning(knob, value); }

int32_t opscale_get_tuning(opscale_tune knob) { return opscale::tuning(knob); }

size_t opscale_linear_workspace_size(int64_t M, int64_t N, int64_t K, opscale_dtype dt) {
  if (M <= 0 || N <= 0 || K <= 0 || !dtype_ok(dt)) return 0;
  return opscale::plan_linear(M, N, K, dt == OPSCALE_BF16, true).ws_bytes;
}

opscale_status opscale_linear(const void* x, const void* W, const void* bias, void* y, int64_t M,
                              int64_t N, int64_t K, opscale_dtype dt, void* workspace, size_t workspace_bytes,
                              hipStream_t stream, opscale_timing* timing) {
  opscale::LinearPlan plan{};
  opscale_status st = check_linear(x, W, bias, y, M, N, K, dt, workspace, workspace_bytes, &plan);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (M == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "linear launch", [&] {
    return opscale::launch_linear(plan, x, W, bias, y, M, N, K, workspace, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_linear(M, N, K, esize(dt), bias != nullptr);
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_swiglu(const void* gate_up, void* out, int64_t M, int64_t F, opscale_dtype dt,
                              hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_swiglu(gate_up, out, M, F, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (M == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "swiglu launch", [&] {
    return opscale::launch_swiglu(gate_up, out, M, F, dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_swiglu(M, F, esize(dt));
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_attn_prefill(const void* q, const void* k, const void* v, int64_t q_row_stride,
                                    int64_t kv_row_stride, void* o, const int32_t* cu_seqlens,
                                    int32_t B, int64_t total_tokens, int32_t max_seqlen, int32_t Hq,
                                    int32_t Hkv, int32_t D, float scale, int32_t causal,
                                    opscale_dtype dt, hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_prefill(q, k, v, q_row_stride, kv_row_stride, o, cu_seqlens, B,
                                    total_tokens, max_seqlen, Hq, Hkv, D, scale, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (B == 0 || total_tokens == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "attn_prefill launch", [&] {
    return opscale::launch_attn_prefill(q, k, v, q_row_stride, kv_row_stride, o, cu_seqlens, B,
                                        total_tokens, max_seqlen, Hq, Hkv, D, scale, causal != 0,
                                        dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    std::vector<int32_t> cu;
    st = copy_ints(cu, cu_seqlens, (int64_t)B + 1, stream);
    if (st != OPSCALE_OK) return st;
    const Work wk = work_prefill(cu, Hq, Hkv, D, esize(dt), causal != 0);
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

size_t opscale_attn_decode_workspace_size(int32_t B, int32_t Hq, int32_t D, int32_t max_context_len) {
  if (B <= 0 || Hq <= 0 || D <= 0) return 16;
  return opscale::decode_workspace_bytes(B, Hq, D, std::max<int32_t>(1, max_context_len));
}

opscale_status opscale_attn_decode(const void* q, int64_t q_row_stride, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* context_lens, void* o,
                                   int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size,
                                   int32_t max_blocks_per_seq, int64_t num_blocks,
                                   int32_t max_context_len, float scale, opscale_dtype dt,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream,
                                   opscale_timing* timing) {
  opscale_status st = check_decode(q, q_row_stride, k_cache, v_cache, block_table, context_lens, o, B, Hq, Hkv, D,
                                   block_size, max_blocks_per_seq, num_blocks, max_context_len,
                                   scale, dt, workspace, workspace_bytes);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (B == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "attn_decode launch", [&] {
    return opscale::launch_attn_decode(q, q_row_stride, k_cache, v_cache, block_table, context_lens, o, B, Hq, Hkv,
                                       D, block_size, max_blocks_per_seq, num_blocks,
                                       max_context_len, scale, dt == OPSCALE_BF16, workspace, stream);
  });
  if (st == OPSCALE_OK && timing) {
    std::vector<int32_t> ctx;
    st = copy_ints(ctx, context_lens, B, stream);
    if (st != OPSCALE_OK) return st;
    const Work wk = work_decode(ctx, Hq, Hkv, D, esize(dt), block_size, max_blocks_per_seq);
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_attn_decode_noalloc(const void* q, int64_t q_row_stride, const void* k_cache,
                                           const void* v_cache, const int32_t* block_table,
                                           const int32_t* context_lens, void* o, int32_t B, int32_t Hq,
                                           int32_t Hkv, int32_t D, int32_t block_size, int32_t max_blocks_per_seq,
                                           int64_t num_blocks, int32_t max_context_len, float scale,
                                           opscale_dtype dt, hipStream_t stream) {
  void* ws = nullptr;
  opscale_status st = static_scratch(&ws);
  if (st != OPSCALE_OK) return st;
  st = check_decode(q, q_row_stride, k_cache, v_cache, block_table, context_lens, o, B, Hq, Hkv, D, block_size,
                    max_blocks_per_seq, num_blocks, max_context_len, scale, dt, ws, kStaticScratchBytes);
  if (st == OPSCALE_ERR_WORKSPACE)
    return fail(OPSCALE_ERR_WORKSPACE, "attn_decode_noalloc: %zu bytes of scratch needed, the library holds %zu",
                opscale::decode_workspace_bytes(B, Hq, D, max_context_len), kStaticScratchBytes);
  if (st != OPSCALE_OK) return st;
  if (B == 0) return OPSCALE_OK;
  const hipError_t e = opscale::launch_attn_decode(q, q_row_stride, k_cache, v_cache, block_table, context_lens, o,
                                                   B, Hq, Hkv, D, block_size, max_blocks_per_seq, num_blocks,
                                                   max_context_len, scale, dt == OPSCALE_BF16, ws, stream);
  return e == hipSuccess ? OPSCALE_OK : hip_fail(e, "attn_decode_noalloc launch");
}

size_t opscale_attn_decode_noalloc_max_bytes(void) { return kStaticScratchBytes; }

opscale_status opscale_rope(void* q, void* k, int64_t q_row_stride, int64_t k_row_stride,
                            const int32_t* positions, int64_t T, int32_t Hq, int32_t Hkv, int32_t D,
                            double theta, opscale_dtype dt, hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_rope(q, k, q_row_stride, k_row_stride, positions, T, Hq, Hkv, D, theta, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (T == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "rope launch", [&] {
    return opscale::launch_rope(q, k, q_row_stride, k_row_stride, positions, T, Hq, Hkv, D, theta,
                                dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_rope(T, Hq, Hkv, D, esize(dt));
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_reshape_and_cache(const void* k, const void* v, int64_t kv_row_stride, void* k_cache,
                                         void* v_cache, const int32_t* slot_mapping, int64_t T, int32_t Hkv,
                                         int32_t D, int32_t block_size, int64_t num_blocks, opscale_dtype dt,
                                         hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_cache_write(k, v, kv_row_stride, k_cache, v_cache, slot_mapping, T, Hkv, D, block_size,
                                        num_blocks, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (T == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "reshape_and_cache launch", [&] {
    return opscale::launch_cache_write(k, v, kv_row_stride, k_cache, v_cache, slot_mapping, T, Hkv, D,
                                       num_blocks * block_size, dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_cache_write(T, Hkv, D, esize(dt));
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_add_rmsnorm(const void* x, void* residual, const void* w, void* y, int64_t M, int64_t H,
                                   float eps, opscale_dtype dt, hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_add_rmsnorm(x, residual, w, y, M, H, eps, dt);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (M == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "add_rmsnorm launch", [&] {
    return opscale::launch_add_rmsnorm(x, residual, w, y, M, H, eps, dt == OPSCALE_BF16, stream);
  });
  if (st == OPSCALE_OK && timing) {
    const Work wk = work_add_rmsnorm(M, H, esize(dt));
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

opscale_status opscale_moe_topk(const float* logits, int32_t* topk_ids, float* topk_weights, int64_t T, int32_t E,
                                int32_t topk, int32_t renormalize, hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_moe_topk(logits, topk_ids, topk_weights, T, E, topk);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (T == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "moe_topk launch", [&] {
    return opscale::launch_moe_topk(logits, topk_ids, topk_weights, T, E, topk, renormalize != 0, stream);
  });
  if (st == OPSCALE_OK && timing) {
    timing->alg_flops = 3.0 * T * E;
    timing->alg_bytes = 4.0 * T * E + 8.0 * T * topk;
  }
  return st;
}

size_t opscale_fused_moe_workspace_size(int64_t T, int32_t H, int32_t F, int32_t E, int32_t topk) {
  return opscale::moe_workspace_bytes(std::max<int64_t>(0, T), std::max(0, H), std::max(0, F), std::max(1, E),
                                      std::max(1, topk));
}

opscale_status opscale_fused_moe(const void* x, const void* w1, const void* w2, const int32_t* topk_ids,
                                 const float* topk_weights, void* out, int64_t T, int32_t H, int32_t F, int32_t E,
                                 int32_t topk, opscale_dtype dt, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream, opscale_timing* timing) {
  opscale_status st = check_fused_moe(x, w1, w2, topk_ids, topk_weights, out, T, H, F, E, topk, dt, workspace,
                                      workspace_bytes);
  if (st != OPSCALE_OK) return st;
  zero_timing(timing);
  if (T == 0) return OPSCALE_OK;
  st = run_timed(stream, timing, "fused_moe launch", [&] {
    return opscale::launch_fused_moe(x, w1, w2, topk_ids, topk_weights, out, T, H, F, E, topk, workspace, stream);
  });
  if (st == OPSCALE_OK && timing) {
    std::vector<int32_t> ids;
    if ((st = copy_ints(ids, topk_ids, T * topk, stream)) != OPSCALE_OK) return st;
    const Work wk = work_fused_moe(ids, T, H, F, E, 2);
    timing->alg_flops = wk.flops;
    timing->alg_bytes = wk.bytes;
  }
  return st;
}

}  // extern "C"

namespace {

// Validates one operator descriptor and binds its launch on `stream` (no
// re-validation per launch); `wk` receives the algorithmic work.
opscale_status prepare_op(const opscale_op_desc* d, hipStream_t stream, const char* who,
                          std::function<hipError_t()>* launch_out, Work* wk_out) {
  const opscale_dtype dt = d->dt;
  opscale_status st = OPSCALE_OK;
  std::function<hipError_t()>& launch = *launch_out;
  Work& wk = *wk_out;
  const bool bf16 = dt == OPSCALE_BF16;
  switch (d->op) {
    case OPSCALE_OP_RMSNORM: {
      const auto& a = d->u.rmsnorm;
      st = check_rmsnorm(a.x, a.w, a.y, a.M, a.H, a.eps, dt);
      if (st != OPSCALE_OK) return st;
      if (a.M == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] { return opscale::launch_rmsnorm(a.x, a.w, a.y, a.M, a.H, a.eps, bf16, stream); };
      wk = work_rmsnorm(a.M, a.H, esize(dt));
      break;
    }
    case OPSCALE_OP_LINEAR: {
      const auto& a = d->u.linear;
      opscale::LinearPlan plan{};
      st = check_linear(a.x, a.W, a.bias, a.y, a.M, a.N, a.K, dt, a.workspace, a.workspace_bytes, &plan);
      if (st != OPSCALE_OK) return st;
      if (a.M == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] { return opscale::launch_linear(plan, a.x, a.W, a.bias, a.y, a.M, a.N, a.K, a.workspace, stream); };
      wk = work_linear(a.M, a.N, a.K, esize(dt), a.bias != nullptr);
      break;
    }
    case OPSCALE_OP_SWIGLU: {
      const auto& a = d->u.swiglu;
      st = check_swiglu(a.gate_up, a.out, a.M, a.F, dt);
      if (st != OPSCALE_OK) return st;
      if (a.M == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] { return opscale::launch_swiglu(a.gate_up, a.out, a.M, a.F, bf16, stream); };
      wk = work_swiglu(a.M, a.F, esize(dt));
      break;
    }
    case OPSCALE_OP_ATTN_PREFILL: {
      const auto& a = d->u.attn_prefill;
      st = check_prefill(a.q, a.k, a.v, a.q_row_stride, a.kv_row_stride, a.o, a.cu_seqlens, a.B,
                         a.total_tokens, a.max_seqlen, a.Hq, a.Hkv, a.D, a.scale, dt);
      if (st != OPSCALE_OK) return st;
      if (a.B == 0 || a.total_tokens == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] {
        return opscale::launch_attn_prefill(a.q, a.k, a.v, a.q_row_stride, a.kv_row_stride, a.o,
                                            a.cu_seqlens, a.B, a.total_tokens, a.max_seqlen, a.Hq,
                                            a.Hkv, a.D, a.scale, a.causal != 0, bf16, stream);
      };
      std::vector<int32_t> cu;
      st = copy_ints(cu, a.cu_seqlens, (int64_t)a.B + 1, stream);
      if (st != OPSCALE_OK) return st;
      wk = work_prefill(cu, a.Hq, a.Hkv, a.D, esize(dt), a.causal != 0);
      break;
    }
    case OPSCALE_OP_ATTN_DECODE: {
      const auto& a = d->u.attn_decode;
      st = check_decode(a.q, a.q_row_stride, a.k_cache, a.v_cache, a.block_table, a.context_lens, a.o, a.B, a.Hq,
                        a.Hkv, a.D, a.block_size, a.max_blocks_per_seq, a.num_blocks,
                        a.max_context_len, a.scale, dt, a.workspace, a.workspace_bytes);
      if (st != OPSCALE_OK) return st;
      if (a.B == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] {
        return opscale::launch_attn_decode(a.q, a.q_row_stride, a.k_cache, a.v_cache, a.block_table, a.context_lens,
                                           a.o, a.B, a.Hq, a.Hkv, a.D, a.block_size,
                                           a.max_blocks_per_seq, a.num_blocks, a.max_context_len,
                                           a.scale, bf16, a.workspace, stream);
      };
      std::vector<int32_t> ctx;
      st = copy_ints(ctx, a.context_lens, a.B, stream);
      if (st != OPSCALE_OK) return st;
      wk = work_decode(ctx, a.Hq, a.Hkv, a.D, esize(dt), a.block_size, a.max_blocks_per_seq);
      break;
    }
    case OPSCALE_OP_ROPE: {
      const auto& a = d->u.rope;
      st = check_rope(a.q, a.k, a.q_row_stride, a.k_row_stride, a.positions, a.T, a.Hq, a.Hkv, a.D, a.theta, dt);
      if (st != OPSCALE_OK) return st;
      if (a.T == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] {
        return opscale::launch_rope(a.q, a.k, a.q_row_stride, a.k_row_stride, a.positions, a.T, a.Hq, a.Hkv, a.D,
                                    a.theta, bf16, stream);
      };
      wk = work_rope(a.T, a.Hq, a.Hkv, a.D, esize(dt));
      break;
    }
    case OPSCALE_OP_RESHAPE_AND_CACHE: {
      const auto& a = d->u.reshape_and_cache;
      st = check_cache_write(a.k, a.v, a.kv_row_stride, a.k_cache, a.v_cache, a.slot_mapping, a.T, a.Hkv, a.D,
                             a.block_size, a.num_blocks, dt);
      if (st != OPSCALE_OK) return st;
      if (a.T == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] {
        return opscale::launch_cache_write(a.k, a.v, a.kv_row_stride, a.k_cache, a.v_cache, a.slot_mapping, a.T,
                                           a.Hkv, a.D, a.num_blocks * a.block_size, bf16, stream);
      };
      wk = work_cache_write(a.T, a.Hkv, a.D, esize(dt));
      break;
    }
    case OPSCALE_OP_ADD_RMSNORM: {
      const auto& a = d->u.add_rmsnorm;
      st = check_add_rmsnorm(a.x, a.residual, a.w, a.y, a.M, a.H, a.eps, dt);
      if (st != OPSCALE_OK) return st;
      if (a.M == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] { return opscale::launch_add_rmsnorm(a.x, a.residual, a.w, a.y, a.M, a.H, a.eps, bf16, stream); };
      wk = work_add_rmsnorm(a.M, a.H, esize(dt));
      break;
    }
    case OPSCALE_OP_FUSED_MOE: {
      const auto& a = d->u.fused_moe;
      st = check_fused_moe(a.x, a.w1, a.w2, a.topk_ids, a.topk_weights, a.out, a.T, a.H, a.F, a.E, a.topk, dt,
                           a.workspace, a.workspace_bytes);
      if (st != OPSCALE_OK) return st;
      if (a.T == 0) return fail(OPSCALE_ERR_INVALID_ARG, "%s: empty problem", who);
      launch = [=] {
        return opscale::launch_fused_moe(a.x, a.w1, a.w2, a.topk_ids, a.topk_weights, a.out, a.T, a.H, a.F, a.E,
                                         a.topk, a.workspace, stream);
      };
      std::vector<int32_t> ids;
      st = copy_ints(ids, a.topk_ids, a.T * a.topk, stream);
      if (st != OPSCALE_OK) return st;
      wk = work_fused_moe(ids, a.T, a.H, a.F, a.E, 2);
      break;
    }
    default:
      return fail(OPSCALE_ERR_INVALID_ARG, "%s: unknown op %d", who, (int)d->op);
  }
  if (!dtype_ok(dt)) return fail(OPSCALE_ERR_INVALID_ARG, "%s: unknown dtype", who);
  return OPSCALE_OK;
}

}  // namespace

extern "C" {

opscale_status opscale_op_profile(const opscale_op_desc* d, int32_t warmup, int32_t iters,
                                  void* flush_buf, size_t flush_bytes, hipStream_t stream,
                                  opscale_profile* out) {
  if (!d || !out) return fail(OPSCALE_ERR_INVALID_ARG, "op_profile: null desc or out");
  if (iters < 1 || warmup < 0) return fail(OPSCALE_ERR_INVALID_ARG, "op_profile: iters must be >= 1, warmup >= 0");
  if (flush_buf && !aligned16(flush_buf)) return fail(OPSCALE_ERR_INVALID_ARG, "op_profile: flush_buf must be 16-byte aligned");
  std::function<hipError_t()> launch;
  Work wk{};
  opscale_status st = prepare_op(d, stream, "op_profile", &launch, &wk);
  if (st != OPSCALE_OK) return st;
  const bool bf16 = d->dt == OPSCALE_BF16;

  hipError_t e = g_events.init();
  if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
  for (int i = 0; i < warmup; ++i) {
    e = launch();
    if (e != hipSuccess) return hip_fail(e, "op_profile warmup launch");
  }
  std::vector<float> us((size_t)iters);
  for (int i = 0; i < iters; ++i) {
    if (flush_buf && flush_bytes) {
      e = opscale::launch_flush(flush_buf, flush_bytes, stream);
      if (e != hipSuccess) return hip_fail(e, "op_profile flush");
    }
    if ((e = hipEventRecord(g_events.start, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if ((e = launch()) != hipSuccess) return hip_fail(e, "op_profile launch");
    if ((e = hipEventRecord(g_events.stop, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if ((e = hipEventSynchronize(g_events.stop)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    if ((e = hipEventElapsedTime(&ms, g_events.start, g_events.stop)) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
    us[(size_t)i] = ms * 1000.f;
  }
  std::vector<float> sorted = us;
  std::sort(sorted.begin(), sorted.end());
  auto pct = [&](double p) {
    const double pos = p * (double)(sorted.size() - 1);
    const size_t lo = (size_t)std::floor(pos), hi = (size_t)std::ceil(pos);
    return (float)(sorted[lo] + (sorted[hi] - sorted[lo]) * (pos - (double)lo));
  };
  double mean = 0;
  for (float x : us) mean += x;
  mean /= (double)us.size();

  // MI355X peaks: bf16 dense matrix 2.5 PFLOP/s, fp32 matrix 157.3 TFLOP/s, HBM 8 TB/s.
  const double peak_flops = bf16 ? 2.5e15 : 157.3e12;
  const double peak_bw = 8.0e12;
  const double t_s = (double)pct(0.5) * 1e-6;
  opscale_profile p{};
  p.iters = iters;
  p.us_median = pct(0.5);
  p.us_p10 = pct(0.1);
  p.us_p90 = pct(0.9);
  p.us_min = sorted.front();
  p.us_mean = (float)mean;
  p.alg_flops = wk.flops;
  p.alg_bytes = wk.bytes;
  p.tflops = t_s > 0 ? wk.flops / t_s * 1e-12 : 0.0;
  p.gbps = t_s > 0 ? wk.bytes / t_s * 1e-9 : 0.0;
  const double ai = wk.bytes > 0 ? wk.flops / wk.bytes : 0.0;
  const double attainable = std::min(peak_flops, ai * peak_bw);
  p.attainable_tflops = attainable * 1e-12;
  p.roofline_frac = attainable > 0 && t_s > 0 ? (wk.flops / t_s) / attainable : 0.0;
  p.bound = ai * peak_bw < peak_flops ? 1 : 0;
  p.weight_bytes = wk.weight;
  p.transient_bytes = wk.transient;
  p.io_bytes = wk.io;
  *out = p;
  return OPSCALE_OK;
}

opscale_status opscale_corun_profile(const opscale_op_desc* a, hipStream_t sa, const opscale_op_desc* b,
                                     hipStream_t sb, int32_t warmup, int32_t iso_iters, float window_ms,
                                     int32_t max_launches, const opscale_corun_trace* trace, opscale_corun* out) {
  if (!a || !b || !out) return fail(OPSCALE_ERR_INVALID_ARG, "corun_profile: null desc or out");
  if (warmup < 0 || iso_iters < 1 || iso_iters > 4096)
    return fail(OPSCALE_ERR_INVALID_ARG, "corun_profile: warmup >= 0 and 1 <= iso_iters <= 4096 required");
  if (max_launches < 4 || max_launches > 8192)
    return fail(OPSCALE_ERR_INVALID_ARG, "corun_profile: max_launches %d outside [4, 8192]", max_launches);
  if (!(window_ms > 0.f && window_ms <= 10000.f))
    return fail(OPSCALE_ERR_INVALID_ARG, "corun_profile: window_ms must be in (0, 10000]");
  if (sa == sb) return fail(OPSCALE_ERR_INVALID_ARG, "corun_profile: the two operators need two streams");
  std::function<hipError_t()> la, lb;
  Work wa{}, wb{};
  opscale_status st = prepare_op(a, sa, "corun_profile (a)", &la, &wa);
  if (st != OPSCALE_OK) return st;
  if ((st = prepare_op(b, sb, "corun_profile (b)", &lb, &wb)) != OPSCALE_OK) return st;
  hipError_t e;
  for (int i = 0; i < warmup; ++i) {
    if ((e = la()) != hipSuccess) return hip_fail(e, "corun warmup launch (a)");
    if ((e = lb()) != hipSuccess) return hip_fail(e, "corun warmup launch (b)");
  }
  if ((e = hipStreamSynchronize(sa)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  if ((e = hipStreamSynchronize(sb)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");

  // T_v(b, p): each operator alone on its stream
  std::vector<float> iso_a, iso_b;
  if ((st = time_loop(la, sa, iso_iters, &iso_a)) != OPSCALE_OK) return st;
  if ((st = time_loop(lb, sb, iso_iters, &iso_b)) != OPSCALE_OK) return st;
  const float ta = median_of(iso_a), tb = median_of(iso_b);
  // the window lasts at least four launches of the slower operator, so that
  // launches of each fit inside the other's span
  const double window_us = std::max((double)window_ms * 1000.0, 4.0 * (double)std::max(ta, tb));
  auto launches = [&](float t_us) {
    const double n = t_us > 0.f ? std::ceil(window_us / (double)t_us) : (double)max_launches;
    return (int)std::max(4.0, std::min((double)max_launches, n));
  };
  const int na = launches(ta), nb = launches(tb);

  // both loops at once: b waits for the reference event recorded on a, and
  // the launches are enqueued in the order of their planned start times
  EventPool pool;
  if ((e = pool.make((size_t)na + (size_t)nb + 3)) != hipSuccess) return hip_fail(e, "hipEventCreate");
  hipEvent_t ref = pool.ev[0];
  hipEvent_t* ea = pool.ev.data() + 1;             // na + 1 events
  hipEvent_t* eb = pool.ev.data() + 2 + (size_t)na;  // nb + 1 events
  if ((e = hipEventRecord(ref, sa)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = hipStreamWaitEvent(sb, ref, 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  if ((e = hipEventRecord(ea[0], sa)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = hipEventRecord(eb[0], sb)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  int ia = 0, ib = 0;
  while (ia < na || ib < nb) {
    const bool take_a = ib >= nb || (ia < na && (double)ia * ta <= (double)ib * tb);
    if (take_a) {
      if ((e = la()) != hipSuccess) return hip_fail(e, "corun launch (a)");
      if ((e = hipEventRecord(ea[++ia], sa)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    } else {
      if ((e = lb()) != hipSuccess) return hip_fail(e, "corun launch (b)");
      if ((e = hipEventRecord(eb[++ib], sb)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
  }
  if ((e = hipEventSynchronize(ea[na])) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  if ((e = hipEventSynchronize(eb[nb])) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  auto stamps = [&](hipEvent_t* ev, int n, std::vector<float>* t) {
    t->resize((size_t)n + 1);
    for (int i = 0; i <= n; ++i) {
      float ms = 0.f;
      const hipError_t r = hipEventElapsedTime(&ms, ref, ev[i]);
      if (r != hipSuccess) return r;
      (*t)[(size_t)i] = ms * 1000.f;
    }
    return hipSuccess;
  };
  std::vector<float> tsa, tsb;
  if ((e = stamps(ea, na, &tsa)) != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
  if ((e = stamps(eb, nb, &tsb)) != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
  // T~_v(b, p): launches wholly inside the other operator's span
  auto inside = [](const std::vector<float>& t, int n, float lo, float hi) {
    std::vector<float> d;
    for (int i = 0; i < n; ++i)
      if (t[(size_t)i] >= lo && t[(size_t)i + 1] <= hi) d.push_back(t[(size_t)i + 1] - t[(size_t)i]);
    return d;
  };
  const std::vector<float> co_a = inside(tsa, na, tsb[0], tsb[(size_t)nb]);
  const std::vector<float> co_b = inside(tsb, nb, tsa[0], tsa[(size_t)na]);
  opscale_corun r{};
  r.n_a = na;
  r.n_b = nb;
  r.overlap_a = (int32_t)co_a.size();
  r.overlap_b = (int32_t)co_b.size();
  r.a_iso_us = ta;
  r.b_iso_us = tb;
  r.a_co_us = median_of(co_a);
  r.b_co_us = median_of(co_b);
  r.interference_a = co_a.empty() || ta <= 0.f ? 0.0 : (double)r.a_co_us / (double)ta;
  r.interference_b = co_b.empty() || tb <= 0.f ? 0.0 : (double)r.b_co_us / (double)tb;
  if (trace) {
    for (int i = 0; i < na; ++i) {
      if (trace->a_start) trace->a_start[i] = tsa[(size_t)i];
      if (trace->a_end) trace->a_end[i] = tsa[(size_t)i + 1];
    }
    for (int i = 0; i < nb; ++i) {
      if (trace->b_start) trace->b_start[i] = tsb[(size_t)i];
      if (trace->b_end) trace->b_end[i] = tsb[(size_t)i + 1];
    }
    for (int i = 0; i < iso_iters; ++i) {
      if (trace->a_iso) trace->a_iso[i] = iso_a[(size_t)i];
      if (trace->b_iso) trace->b_iso[i] = iso_b[(size_t)i];
    }
  }
  *out = r;
  return OPSCALE_OK;
}

}  // extern "C"
