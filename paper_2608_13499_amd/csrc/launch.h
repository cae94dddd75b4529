// Host-side launchers of the gfx950 kernels.  Arguments are validated by the
// C ABI layer (abi.hip) before any of these is called; each launcher only
// sizes the grid and enqueues on `s`, returning the launch status.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "opscale.h"

namespace opscale {

// Process-wide tuning and test overrides set through opscale_set_tuning;
// -1 means automatic (the shape decides).
int32_t tuning(opscale_tune knob);

hipError_t launch_rmsnorm(const void* x, const void* w, void* y, int64_t M, int64_t H, float eps,
                          bool bf16, hipStream_t s);

hipError_t launch_swiglu(const void* gu, void* out, int64_t M, int64_t F, bool bf16, hipStream_t s);

// The path of one linear call: which kernel, which tile, how K is split and
// how much caller workspace the split partials need.  split_ok == false
// plans only paths that need no workspace.  The workspace query and the
// launch both take it from plan_linear, so they always agree.
struct LinearPlan {
  enum Path { kF32 = 0, kSkinny = 1, kTiled = 2, kDecode = 3 };
  int path;
  int cfg;          // tiled: which block tile (k_gemm.hip)
  int splits;       // > 1: every tile split over K (partials [splits, M, N] fp32)
  int tail_splits;  // > 1: only the last partial round split over K
  size_t ws_bytes;  // workspace the partials need (0: none)
};
LinearPlan plan_linear(int64_t M, int64_t N, int64_t K, bool bf16, bool split_ok);
hipError_t launch_linear(const LinearPlan& plan, const void* x, const void* W, const void* bias, void* y, int64_t M,
                         int64_t N, int64_t K, void* ws, hipStream_t s);

// Grouped bf16 GEMM of a mixture-of-experts layer: output rows grouped by
// expert (expert e owns rows [rows[e], rows[e+1]) and tile-rows [tiles[e],
// tiles[e+1]) of tile_rows rows); row m multiplies x row gather[m] (m if
// gather is null) by W + e * w_stride ([N, K] per expert).  max_rows bounds
// rows[E]; y has max_rows rows of N.  tile_rows is
// grouped_gemm_tile_rows(max_rows, E), the value the tile table was built with.
int32_t grouped_gemm_tile_rows(int64_t rows, int32_t E);
// swiglu_f > 0: W is a gate-up weight [2F, K] (N = 2F) and y receives
// silu(gate) * up, [rows, F] (fused epilogue); every expert's W must then span
// less than 4 GB.
hipError_t launch_gemm_grouped(const void* x, int64_t x_rows, const void* W, int64_t w_stride, void* y,
                               int64_t max_rows, int64_t N, int64_t K, int32_t E, int32_t tile_rows,
                               const int32_t* gather, const int32_t* rows, const int32_t* tiles, int32_t swiglu_f,
                               hipStream_t s);

// The small-M (decode batch) bf16 linear: all M rows per workgroup, K split
// over its waves.  Supported for 1 <= M <= kSkinnyMaxM with K % 32 == 0;
// preferred over the tiled GEMM where it measured faster.
constexpr int64_t kSkinnyMaxM = 256;
bool skinny_linear_supported(int64_t M, int64_t N, int64_t K);
bool skinny_linear_preferred(int64_t M, int64_t N, int64_t K);
hipError_t launch_linear_skinny(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, hipStream_t s);

// The decode-batch bf16 linear (k_gemm_decode.hip): 128 output columns and
// all M rows per workgroup, the weights streamed into registers, K split
// over workgroups up to about one per CU (fp32 partials [splits, M, N] in the
// workspace, then launch_splitk_reduce).  Supported for 1 <= M <=
// kDecodeMaxM with K % 64 == 0.
constexpr int64_t kDecodeMaxM = 256;
bool decode_linear_supported(int64_t M, int64_t N, int64_t K);
int decode_linear_splits(int64_t M, int64_t N, int64_t K);
size_t decode_linear_ws_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_linear_decode(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, int splits, void* ws, hipStream_t s);
// y[m][n] = bf16(sum over s < splits of part[s][m][n], in split order, +
// bias[n]); N % 8 == 0.
hipError_t launch_splitk_reduce(const float* part, int splits, const void* bias, void* y, int64_t M, int64_t N,
                                hipStream_t s);

hipError_t launch_attn_prefill(const void* q, const void* k, const void* v, int64_t q_stride,
                               int64_t kv_stride, void* o, const int32_t* cu, int32_t B,
                               int64_t total_tokens, int32_t max_seqlen, int32_t Hq, int32_t Hkv,
                               int32_t D, float scale, bool causal, bool bf16, hipStream_t s);

// Balanced split-KV decode: workgroups of a launch (each takes an equal range
// of the batch's 32-key tiles) and the workspace it needs (the tile prefix
// sums, then (workgroups + B) x Hq partial results of D + 2 floats).
int32_t decode_workgroups(int32_t B, int32_t max_context_len, int32_t groups);
size_t decode_workspace_bytes(int32_t B, int32_t Hq, int32_t D, int32_t max_context_len);

hipError_t launch_attn_decode(const void* q, int64_t q_stride, const void* kc, const void* vc, const int32_t* table,
                              const int32_t* ctx, void* o, int32_t B, int32_t Hq, int32_t Hkv,
                              int32_t D, int32_t block_size, int32_t max_blocks, int64_t num_blocks,
                              int32_t max_context_len, float scale, bool bf16, void* ws,
                              hipStream_t s);

// Rotary embedding of the q and k heads in place (rows of q_stride /
// k_stride elements, token t at position pos[t]).
hipError_t launch_rope(void* q, void* k, int64_t q_stride, int64_t k_stride, const int32_t* pos, int64_t T,
                       int32_t Hq, int32_t Hkv, int32_t D, double theta, bool bf16, hipStream_t s);

// K/V rows of T tokens to cache rows slots[t] (skipped outside [0, num_slots)).
hipError_t launch_cache_write(const void* k, const void* v, int64_t kv_stride, void* kc, void* vc,
                              const int32_t* slots, int64_t T, int32_t Hkv, int32_t D, int64_t num_slots,
                              bool bf16, hipStream_t s);

// residual <- x + residual; y <- rmsnorm(residual) * w.
hipError_t launch_add_rmsnorm(const void* x, void* res, const void* w, void* y, int64_t M, int64_t H, float eps,
                              bool bf16, hipStream_t s);

// Mixture-of-experts: top-k routing and the fused expert MLPs (k_moe.hip).
int32_t moe_max_experts();
size_t moe_workspace_bytes(int64_t T, int32_t H, int32_t F, int32_t E, int32_t topk);
hipError_t launch_moe_topk(const float* logits, int32_t* ids, float* wts, int64_t T, int32_t E, int32_t k,
                           bool renormalize, hipStream_t s);
hipError_t launch_fused_moe(const void* x, const void* w1, const void* w2, const int32_t* ids, const float* wts,
                            void* out, int64_t T, int32_t H, int32_t F, int32_t E, int32_t k, void* ws,
                            hipStream_t s);

// Reads `bytes` of `buf` through the caches (evicts L2 and the last-level
// cache, leaving only clean lines, before a timed iteration).
hipError_t launch_flush(void* buf, size_t bytes, hipStream_t s);

}  // namespace opscale
