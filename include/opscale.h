/*
 * opscale.h -- C ABI of the per-operator decoder-layer forward for AMD MI355X
 * (CDNA4, gfx950).
 *
 * The paper treats an LLM as a dataflow of operators that are profiled,
 * provisioned and scaled one by one (Section 2.2 "Rethinking the Scaling
 * Unit"; Section 4.2 "Operator Profiling").  Each entry point below is one such
 * operator of a Llama-style decoder layer: RMS Norm, the QKV / O / gate-up /
 * down linears, the fused SiLU-multiply activation, causal grouped-query
 * prefill attention over a ragged batch of prompts, and decode attention over a
 * paged KV cache.  Every call can return its kernel-only device time, measured
 * with device events around the launches and excluding host overhead (Section
 * 2.1 "Compute Sensitivity"), together with the operator's algorithmic flops
 * and bytes, the inputs of the profiler's T_v / M_v / C_v tables (Section 3.1,
 * Section 4.2).
 *
 * Conventions shared by every entry point
 *  - Pointers: all tensor pointers are DEVICE pointers to caller-owned memory,
 *    16-byte aligned.  The library never allocates or frees device memory in an
 *    operator call: every scratch buffer (the linear's split-K partials, the
 *    decode split-KV partials, the mixture-of-experts intermediates) is a
 *    caller workspace whose size a *_workspace_size query returns.
 *  - Layout: row-major, innermost dimension contiguous.  Element type is given
 *    by `dt` and shared by every tensor of the call (indices are int32).
 *  - Sizes: int64 element counts.  A zero-sized problem (M == 0, B == 0 or
 *    total_tokens == 0) is a successful no-op.  Negative sizes are invalid.
 *  - Streams: work is enqueued on `stream` (0 = the null stream).  With
 *    `timing == NULL` a call is fully asynchronous.  With `timing != NULL` the
 *    call records two device events on `stream` around its launches, waits for
 *    the second, and fills the struct (a blocking call).
 *  - Errors: a call validates every argument before enqueuing anything and
 *    returns OPSCALE_ERR_INVALID_ARG / _UNSUPPORTED / _WORKSPACE with nothing
 *    enqueued.  A failed HIP call returns OPSCALE_ERR_HIP.  The thread-local
 *    message of the last failure is available from opscale_last_error().
 *    Nothing aborts, exits or throws across this interface.
 *  - Concurrency: entry points are re-entrant; the only library state is a
 *    pair of timing events per host thread, created on first use, and the
 *    process-wide tuning overrides of opscale_set_tuning (all automatic
 *    unless a caller sets one).
 */
#ifndef OPSCALE_H
#define OPSCALE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OPSCALE_OK = 0,
  OPSCALE_ERR_INVALID_ARG = 1, /* null pointer, bad size, misalignment */
  OPSCALE_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. head_dim 96) */
  OPSCALE_ERR_WORKSPACE = 3,   /* caller workspace smaller than required */
  OPSCALE_ERR_HIP = 4          /* a HIP runtime call or launch failed */
} opscale_status;

typedef enum {
  OPSCALE_F32 = 0,  /* fp32 storage, fp32 arithmetic */
  OPSCALE_BF16 = 1  /* bf16 storage, fp32 accumulation, bf16 result */
} opscale_dtype;

/* Kernel-only time of one call plus its algorithmic work: flops counted as
 * 2 per multiply-add of the contractions, bytes as every input read once and
 * every output written once (weights once, K/V once per KV head, causal
 * attention over the visible lower triangle only). */
typedef struct {
  float elapsed_us;
  double alg_flops;
  double alg_bytes;
} opscale_timing;

/*
 * Tuning and test overrides.  Not needed in normal use: every knob starts at
 * -1, "automatic", and each entry point then picks its kernel path from the
 * problem shape.  Tests and tuning sweeps force one path with another value.
 * A setting is process-wide and applies to calls made after it; calls in
 * flight keep the path they were planned with.  A workspace size queried
 * under one setting is valid for calls made under the same setting.
 * Returns OPSCALE_ERR_INVALID_ARG for an unknown knob or a value out of range.
 */
typedef enum {
  OPSCALE_TUNE_GEMM_TILE = 0,        /* bf16 linear block tile: 0 = 256x256 (four waves), 1 = 192x256,
                                        2 = 256x128, 3 = 256x256 as eight waves (forcing one also turns
                                        off the small-M and split-K paths) */
  OPSCALE_TUNE_GEMM_SKINNY = 1,      /* 0: never the small-M kernel; 1: wherever it is supported */
  OPSCALE_TUNE_GEMM_SPLITK = 2,      /* 0: no K split for decode-sized M */
  OPSCALE_TUNE_GEMM_TAIL = 3,        /* 0: no K split of the last partly filled round */
  OPSCALE_TUNE_SKINNY_NG = 4,        /* 1 or 2: 16 or 32 output columns per small-M workgroup */
  OPSCALE_TUNE_PREFILL_SCHEDULE = 5, /* 0: one workgroup per grid cell; 1: the work list */
  OPSCALE_TUNE_MOE_FUSE = 6,         /* 0: gate-up output, then the SwiGLU kernel */
  OPSCALE_TUNE_GEMM_DECODE = 7,      /* 0: never the decode-batch kernel; 1: wherever it is supported */
  OPSCALE_TUNE_COUNT = 8
} opscale_tune;
opscale_status opscale_set_tuning(opscale_tune knob, int32_t value);
/* The current value of a knob (-1: automatic, also for an unknown knob). */
int32_t opscale_get_tuning(opscale_tune knob);

/* Library version string, e.g. "opscale 0.1.0 gfx950". */
const char* opscale_version(void);
const char* opscale_status_string(opscale_status s);
/* Message of the last failed call on this host thread ("" if none). */
const char* opscale_last_error(void);

/*
 * RMS Norm (Section 2.1: the memory-bound, compute-light operator).
 *   y[m, j] = x[m, j] / sqrt(mean_j x[m, j]^2 + eps) * w[j]
 * x, y: [M, H]; w: [H].  Sum of squares in fp32, one rounding at the output.
 * In-place (y == x) is allowed.  H * sizeof(dt) must be a multiple of 16.
 */
opscale_status opscale_rmsnorm(const void* x, const void* w, void* y, int64_t M, int64_t H,
                               float eps, opscale_dtype dt, hipStream_t stream,
                               opscale_timing* timing);

/*
 * Bytes of device workspace opscale_linear can use for these sizes: the fp32
 * partial results of a K split (small M, or the last partly filled round of
 * tiles of a large problem).  0 when the planned path splits nothing.
 */
size_t opscale_linear_workspace_size(int64_t M, int64_t N, int64_t K, opscale_dtype dt);

/*
 * Linear projection (Section 2.1: QKV Linear, wide projections, MLP linears).
 *   y[m, n] = sum_k x[m, k] * W[n, k] (+ bias[n])
 * x: [M, K]; W: [N, K] (the nn.Linear weight layout); bias: [N] or NULL;
 * y: [M, N], must not alias x or W.  bf16: MFMA with fp32 accumulation.
 * K * sizeof(dt) and N * sizeof(dt) must be multiples of 16.
 * The bf16 path (small-M kernel, decode-batch kernel for 33-128 rows, or a
 * 256x256, 192x256 or 256x128 block tile, with K split over workgroups where
 * that fills the GPU) is chosen per shape.
 * workspace: NULL, or DEVICE scratch of workspace_bytes, 16-byte aligned, not
 *   overlapping x, W or y.  NULL takes a path that needs none (no K split;
 *   slower for decode-sized M and for a last round of tiles that is mostly
 *   idle).  Non-NULL must hold opscale_linear_workspace_size(M, N, K, dt)
 *   bytes, else OPSCALE_ERR_WORKSPACE with nothing enqueued.  Its contents on
 *   entry are ignored; calls sharing a workspace must be stream-ordered.
 *   Split partials are summed in a fixed order, so results are deterministic.
 */
opscale_status opscale_linear(const void* x, const void* W, const void* bias, void* y,
                              int64_t M, int64_t N, int64_t K, opscale_dtype dt,
                              void* workspace, size_t workspace_bytes,
                              hipStream_t stream, opscale_timing* timing);

/*
 * Fused SiLU-and-multiply, the SwiGLU activation ("act_and_mul" / "SiLu Mul",
 * Section 2.1 memory study and Appendix C).
 *   out[m, f] = silu(gate_up[m, f]) * gate_up[m, F + f],  silu(z) = z / (1 + e^-z)
 * gate_up: [M, 2F] (gate half first: the merged gate-up linear's output);
 * out: [M, F].  fp32 arithmetic.  F * sizeof(dt) must be a multiple of 16.
 */
opscale_status opscale_swiglu(const void* gate_up, void* out, int64_t M, int64_t F,
                              opscale_dtype dt, hipStream_t stream, opscale_timing* timing);

/*
 * Prefill self-attention over a ragged batch (Section 2.1: quadratic in prompt
 * length, FlashAttention-style with no stored score matrix; grouped-query
 * attention as in the Table 3 models).
 * For prompt b (tokens cu_seqlens[b] .. cu_seqlens[b+1]-1), local query i,
 * query head h and KV head g = h / (Hq / Hkv):
 *   o[t, h, :] = sum_{j visible} softmax_j(scale * q[t, h, :] . k[c_b + j, g, :]) v[c_b + j, g, :]
 * where key j is visible iff j <= i (causal != 0) or j < L_b (causal == 0).
 * q: token t, head h at q + t * q_row_stride + h * D (elements); k and v: token t,
 *   KV head g at k/v + t * kv_row_stride + g * D.  The strides let q, k, v be
 *   views into the packed output of the QKV linear.
 * o: [total_tokens, Hq, D] contiguous.
 * cu_seqlens: DEVICE int32 [B + 1], cu_seqlens[0] = 0, non-decreasing,
 *   cu_seqlens[B] = total_tokens.  Zero-length prompts are allowed.
 * max_seqlen: an upper bound on the prompt lengths, used to size the launch;
 *   the result does not depend on it being tight (it must be >= 1).
 * scale must be finite and > 0 (1/sqrt(D) for standard attention).
 * D must be 64 or 128; Hkv must divide Hq.  bf16: QK^T and PV on MFMA, fp32
 *   online softmax, probabilities rounded to bf16 for the PV product.
 */
opscale_status opscale_attn_prefill(const void* q, const void* k, const void* v,
                                    int64_t q_row_stride, int64_t kv_row_stride, void* o,
                                    const int32_t* cu_seqlens, int32_t B, int64_t total_tokens,
                                    int32_t max_seqlen, int32_t Hq, int32_t Hkv, int32_t D,
                                    float scale, int32_t causal, opscale_dtype dt,
                                    hipStream_t stream, opscale_timing* timing);

/*
 * Bytes of device workspace that opscale_attn_decode needs for these sizes
 * (split-KV partial results).  0 is never returned for B > 0.
 */
size_t opscale_attn_decode_workspace_size(int32_t B, int32_t Hq, int32_t D,
                                          int32_t max_context_len);

/*
 * Decode attention, one new query token per sequence, over a paged KV cache
 * (Section 2.1 decode phase; Appendix E: decode is memory-bound; the serving
 * engine of Section 5 keeps K/V in a paged cache).
 *   o[b, h, :] = sum_{j < n_b} softmax_j(scale * q[b, h, :] . K_b[j, g, :]) V_b[j, g, :]
 * with n_b = context_lens[b] (already including the new token, whose K/V were
 * written to the cache beforehand) and K_b[j] = k_cache[block_table[b, j / bs], j % bs].
 * q: [B, Hq, D] rows of q_row_stride elements (>= Hq * D, a multiple of 16
 * bytes; a view into the QKV linear's output is fine); o: [B, Hq, D] dense;
 * k_cache, v_cache: [num_blocks, block_size, Hkv, D];
 * block_table: DEVICE int32 [B, max_blocks_per_seq]; context_lens: DEVICE int32 [B].
 * A context length of 0 yields a zero output row.  Lengths above
 * max_blocks_per_seq * block_size are clamped to it.  Keys whose block id is
 * outside [0, num_blocks) are skipped (never read); a row whose keys are all
 * skipped is zero.
 * max_context_len: the expected largest context length; it sizes the
 *   split-KV launch (one workgroup per 32 keys of B x max_context_len, at most
 *   256, each taking an equal share of the keys actually present) and the
 *   workspace.  Longer contexts are still served whole; the value changes
 *   only how the keys are split, so results agree to rounding across values.
 * workspace: DEVICE scratch of at least opscale_attn_decode_workspace_size(B,
 *   Hq, D, max_context_len) bytes, else OPSCALE_ERR_WORKSPACE.  Contents on
 *   entry are ignored.  Calls sharing a workspace must be stream-ordered.
 * scale must be finite and > 0.  block_size must be a power of two in
 *   [1, 1024]; D 64 or 128; Hkv | Hq; on the bf16 path Hq / Hkv is 1, 2, 4 or 8.
 */
opscale_status opscale_attn_decode(const void* q, int64_t q_row_stride, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* context_lens,
                                   void* o, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                   int32_t block_size, int32_t max_blocks_per_seq,
                                   int64_t num_blocks, int32_t max_context_len, float scale,
                                   opscale_dtype dt, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream, opscale_timing* timing);

/*
 * opscale_attn_decode without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same operation, arguments, layouts and
 * kernels as opscale_attn_decode (and bitwise the same output); the split-KV
 * partials go to a scratch array the library holds in device memory, one copy
 * per GPU it runs on, kept until the process ends
 * (opscale_attn_decode_noalloc_max_bytes() bytes, 64 MiB).  No device memory
 * is allocated or freed, and no timing is taken (the call is asynchronous).
 *  - Sizes whose opscale_attn_decode_workspace_size(B, Hq, D,
 *    max_context_len) exceeds that maximum return OPSCALE_ERR_WORKSPACE with
 *    nothing enqueued (e.g. B = 1024, Hq = 64, D = 128 needs 42.6 MB: fits).
 *  - Every call on one GPU shares that GPU's array: calls that overlap in
 *    time on one GPU (on different streams, or from different host threads)
 *    race on it and must be ordered by the caller.  Nothing in the array needs
 *    to start at zero; each call writes what it later reads.
 */
opscale_status opscale_attn_decode_noalloc(const void* q, int64_t q_row_stride, const void* k_cache,
                                           const void* v_cache, const int32_t* block_table,
                                           const int32_t* context_lens, void* o, int32_t B, int32_t Hq,
                                           int32_t Hkv, int32_t D, int32_t block_size, int32_t max_blocks_per_seq,
                                           int64_t num_blocks, int32_t max_context_len, float scale,
                                           opscale_dtype dt, hipStream_t stream);
/* Bytes of the scratch array opscale_attn_decode_noalloc uses (its size limit). */
size_t opscale_attn_decode_noalloc_max_bytes(void);

/* ---------------------------------------------------------------------------
 * The operators around attention in a full decoder layer.
 * ------------------------------------------------------------------------- */

/*
 * Rotary position embedding of the query and key heads, in place (the RoPE
 * attention operator that Section 5.6 lists among those shared by Llama-family
 * models), rotate-half form.  For token t at position p = positions[t] and
 * pair i < D/2 of every head, with inverse frequency f_i = theta^(-2i/D) and
 * angle a = p * f_i:
 *   x[i] <- x[i] cos a - x[i + D/2] sin a,   x[i + D/2] <- x[i + D/2] cos a + x[i] sin a.
 * q: [T, Hq, D] rows of q_row_stride elements; k: [T, Hkv, D] rows of
 * k_row_stride elements (both may be views into the QKV linear's output);
 * positions: device int32 [T].  The angle is formed and reduced modulo 2 pi
 * in fp64.  D 64 or 128; theta finite and > 0; q and k must not share heads.
 * 16-byte aligned q and k, strides multiples of 16 bytes.
 */
opscale_status opscale_rope(void* q, void* k, int64_t q_row_stride, int64_t k_row_stride,
                            const int32_t* positions, int64_t T, int32_t Hq, int32_t Hkv, int32_t D,
                            double theta, opscale_dtype dt, hipStream_t stream, opscale_timing* timing);

/*
 * Paged KV-cache write (the reshape_and_cache operator of Section 2.1's
 * memory study): the K and V rows of token t go to cache row
 * slot_mapping[t], i.e. block slot / block_size, offset slot % block_size of
 * k_cache and v_cache [num_blocks, block_size, Hkv, D].  A token whose slot is
 * outside [0, num_blocks * block_size) is skipped (padding).
 * k, v: [T, Hkv, D] rows of kv_row_stride elements (views into the QKV output
 * are fine); slot_mapping: device int32 [T]; num_blocks * block_size < 2^31.
 * The caches must not overlap k or v.  Tokens sharing a slot race.
 */
opscale_status opscale_reshape_and_cache(const void* k, const void* v, int64_t kv_row_stride, void* k_cache,
                                         void* v_cache, const int32_t* slot_mapping, int64_t T, int32_t Hkv,
                                         int32_t D, int32_t block_size, int64_t num_blocks, opscale_dtype dt,
                                         hipStream_t stream, opscale_timing* timing);

/*
 * Residual add fused with RMS Norm, the form each norm of a decoder layer
 * takes after the first: residual <- x + residual (rounded once to dt) and
 * y <- (x + residual) / sqrt(mean((x + residual)^2) + eps) * w, the norm taken
 * of the unrounded fp32 sum.  x, residual, y: [M, H]; w: [H].  y may be x;
 * residual must not overlap x, y or w.  Same size rules as opscale_rmsnorm,
 * and a row is at most 16 KB (H <= 8192 in bf16), else OPSCALE_ERR_UNSUPPORTED.
 */
opscale_status opscale_add_rmsnorm(const void* x, void* residual, const void* w, void* y, int64_t M, int64_t H,
                                   float eps, opscale_dtype dt, hipStream_t stream, opscale_timing* timing);

/* ---------------------------------------------------------------------------
 * Operator profiling (Section 4.2 "Operator Profiling": per-operator compute
 * time T_v and memory M_v; Appendix C "Dataflow Characteristics": the payload
 * an operator hands to the next one, the basis of C_v).
 * ------------------------------------------------------------------------- */
typedef enum {
  OPSCALE_OP_RMSNORM = 0,
  OPSCALE_OP_LINEAR = 1,
  OPSCALE_OP_SWIGLU = 2,
  OPSCALE_OP_ATTN_PREFILL = 3,
  OPSCALE_OP_ATTN_DECODE = 4,
  OPSCALE_OP_ROPE = 5,
  OPSCALE_OP_RESHAPE_AND_CACHE = 6,
  OPSCALE_OP_ADD_RMSNORM = 7,
  OPSCALE_OP_FUSED_MOE = 8
} opscale_op;

/* One operator call: the argument list of the matching entry point. */
typedef struct {
  opscale_op op;
  opscale_dtype dt;
  union {
    struct { const void* x; const void* w; void* y; int64_t M, H; float eps; } rmsnorm;
    struct {
      const void* x; const void* W; const void* bias; void* y; int64_t M, N, K;
      void* workspace; size_t workspace_bytes;
    } linear;
    struct { const void* gate_up; void* out; int64_t M, F; } swiglu;
    struct {
      const void *q, *k, *v; int64_t q_row_stride, kv_row_stride; void* o;
      const int32_t* cu_seqlens; int32_t B; int64_t total_tokens; int32_t max_seqlen;
      int32_t Hq, Hkv, D; float scale; int32_t causal;
    } attn_prefill;
    struct {
      const void* q; int64_t q_row_stride; const void *k_cache, *v_cache;
      const int32_t *block_table, *context_lens; void* o;
      int32_t B, Hq, Hkv, D, block_size, max_blocks_per_seq; int64_t num_blocks;
      int32_t max_context_len; float scale; void* workspace; size_t workspace_bytes;
    } attn_decode;
    struct {
      void *q, *k; int64_t q_row_stride, k_row_stride; const int32_t* positions; int64_t T;
      int32_t Hq, Hkv, D; double theta;
    } rope;
    struct {
      const void *k, *v; int64_t kv_row_stride; void *k_cache, *v_cache; const int32_t* slot_mapping;
      int64_t T; int32_t Hkv, D, block_size; int64_t num_blocks;
    } reshape_and_cache;
    struct { const void* x; void* residual; const void* w; void* y; int64_t M, H; float eps; } add_rmsnorm;
    struct {
      const void *x, *w1, *w2; const int32_t* topk_ids; const float* topk_weights; void* out;
      int64_t T; int32_t H, F, E, topk; void* workspace; size_t workspace_bytes;
    } fused_moe;
  } u;
} opscale_op_desc;

typedef struct {
  int32_t iters;
  float us_median, us_p10, us_p90, us_min, us_mean;
  double alg_flops, alg_bytes;
  double tflops;          /* alg_flops / median time, in TFLOP/s */
  double gbps;            /* alg_bytes / median time, in GB/s (1e9) */
  double attainable_tflops; /* min(compute peak, flops/byte * HBM peak) */
  double roofline_frac;   /* tflops / attainable_tflops */
  int32_t bound;          /* 0: matrix-core bound, 1: HBM bound */
  int64_t weight_bytes;   /* M_v, static part: parameters */
  int64_t transient_bytes;/* M_v, transient part: activations / KV touched */
  int64_t io_bytes;       /* output payload passed to the next operator */
} opscale_profile;

/*
 * Run the described operator `warmup` times untimed, then `iters` times, each
 * preceded (when flush_buf != NULL) by a device read of flush_bytes of
 * flush_buf, so that no operand is served from L2 or the 256 MB last-level
 * cache and no dirty line is left for the operator to write back
 * (flush_buf's contents are don't-care).
 * Each iteration is timed alone with device events.  Fills `out` with the
 * timing distribution, the algorithmic work and the roofline fraction against
 * MI355X peaks (bf16 matrix 2.5 PFLOP/s, fp32 matrix 157.3 TFLOP/s, HBM
 * 8 TB/s).  Blocking.  iters must be >= 1.
 */
opscale_status opscale_op_profile(const opscale_op_desc* desc, int32_t warmup, int32_t iters,
                                  void* flush_buf, size_t flush_bytes, hipStream_t stream,
                                  opscale_profile* out);

/* ---------------------------------------------------------------------------
 * Peak probes: what this GPU's matrix cores and HBM deliver, measured, to
 * report the operators against beside the published peaks (the paper
 * characterizes each operator by how much of the GPU it uses, Section 2.1).
 * Blocking; results are means over reps launches after one untimed launch.
 * ------------------------------------------------------------------------- */

/*
 * bf16 MFMA throughput: 4 waves per SIMD on every CU, each running 8
 * independent chains of iters 16x16x32 bf16 MFMAs on register operands
 * (non-zero values); iters is rounded up to a multiple of 4.  *tflops =
 * flops / time.  1 <= iters <= 2^24, 1 <= reps <= 1000.
 */
opscale_status opscale_probe_mfma(int64_t iters, int32_t reps, hipStream_t stream, double* tflops);

/*
 * HBM streaming: with dst NULL, read `bytes` of src (DEVICE, 16-byte aligned)
 * once per launch with 16-byte nontemporal loads (*gbps = bytes / time); with
 * dst (DEVICE, `bytes`, not overlapping src) copy src to dst (*gbps =
 * 2 * bytes / time).  Use a buffer well above the 256 MB last-level cache.
 * bytes a multiple of 16; 1 <= reps <= 1000.
 */
opscale_status opscale_probe_hbm(const void* src, void* dst, size_t bytes, int32_t reps, hipStream_t stream,
                                 double* gbps);

/* ---------------------------------------------------------------------------
 * Mixture-of-experts FFN (the FusedMoE operator of the paper's MoE models,
 * Qwen2-57B-A14B and Mixtral-8x7B: Table 3; Section 2.1 counts it among the
 * compute-heavy linear operators, Appendix D shows it dominating at short
 * sequences).
 * ------------------------------------------------------------------------- */

/*
 * Top-k routing: for each of T tokens, the topk experts with the largest
 * logits (logits: DEVICE fp32 [T, E], finite), listed by decreasing logit,
 * the lower expert index first among equal logits; topk_weights[t, j] is the
 * softmax of the token's E logits at expert topk_ids[t, j] (fp32), divided by
 * the sum over the topk picks when renormalize != 0.  topk_ids: DEVICE int32
 * [T, topk]; topk_weights: DEVICE fp32 [T, topk].
 * 1 <= E <= 1024, 1 <= topk <= min(E, 16).
 */
opscale_status opscale_moe_topk(const float* logits, int32_t* topk_ids, float* topk_weights, int64_t T,
                                int32_t E, int32_t topk, int32_t renormalize, hipStream_t stream,
                                opscale_timing* timing);

/* Bytes of device workspace opscale_fused_moe needs for these sizes. */
size_t opscale_fused_moe_workspace_size(int64_t T, int32_t H, int32_t F, int32_t E, int32_t topk);

/*
 * The routed expert MLPs:
 *   out[t] = sum_j topk_weights[t, j] * W2[e] (silu(W1g[e] x[t]) * (W1u[e] x[t])),
 *   e = topk_ids[t, j],
 * with W1[e] = [W1g; W1u] ([2F, H]: the F gate rows first, as in the dense
 * gate-up linear) and W2[e] [H, F].  x: [T, H]; w1: [E, 2F, H]; w2: [E, H, F];
 * out: [T, H] (bf16, must not overlap x); topk_ids: DEVICE int32 [T, topk]
 * (an id outside [0, E) contributes nothing); topk_weights: DEVICE fp32
 * [T, topk].  bf16 only (OPSCALE_ERR_UNSUPPORTED otherwise); H and F
 * multiples of 8; 1 <= E <= 1024; 1 <= topk <= 64; T * H and
 * T * topk * 2F below 2^30 (else OPSCALE_ERR_UNSUPPORTED).
 * The token-expert pairs are sorted by expert (stable) and each expert's rows
 * run through two grouped GEMMs (gate-up with the SwiGLU, then down, rounded
 * to bf16 as the dense layer's intermediates are); the topk results of a
 * token are summed in fp32 in slot order.  Deterministic.
 * workspace: DEVICE, at least opscale_fused_moe_workspace_size(...) bytes,
 * 16-byte aligned, else OPSCALE_ERR_WORKSPACE; calls sharing one must be
 * stream-ordered.
 */
opscale_status opscale_fused_moe(const void* x, const void* w1, const void* w2, const int32_t* topk_ids,
                                 const float* topk_weights, void* out, int64_t T, int32_t H, int32_t F,
                                 int32_t E, int32_t topk, opscale_dtype dt, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream, opscale_timing* timing);

/* ---------------------------------------------------------------------------
 * Spatial sharing: operators on disjoint sets of compute units.
 *
 * The paper runs colocated operators on separate streams that each own a
 * share p of the GPU's SMs (Section 2.1's SM-allocation sensitivity; the
 * interference model of Section 4.4, Eq. 5, validated in Section 5.7,
 * Table 2).  On MI355X the
 * equivalent is a stream whose CU mask selects the compute units its kernels
 * may use.  The GPU has 256 CUs in 8 XCDs, and each XCD has its own L2 and
 * receives every 8th workgroup, so a share is laid out evenly over the XCDs.
 * ------------------------------------------------------------------------- */

/*
 * The current device's CU count, XCD count, and how the bits of a stream's
 * CU mask map to XCDs: interleaved = 1 when mask bit n is CU n / num_xcds of
 * XCD n % num_xcds, 0 when it is CU n % (num_cus / num_xcds) of XCD
 * n / (num_cus / num_xcds).  The mapping is measured once per device, at the
 * first call, by running opscale_cu_probe on a stream masked to the first
 * num_cus / num_xcds bits (blocking).  That first call is set-up, not an
 * operator call: it allocates and frees an 8-byte-per-workgroup result buffer
 * for the probe and creates and destroys the masked stream; later calls touch
 * the device not at all.  OPSCALE_ERR_UNSUPPORTED if the probe matches neither
 * mapping.
 */
opscale_status opscale_cu_layout(int32_t* num_cus, int32_t* num_xcds, int32_t* interleaved);

/*
 * Host only (no device needed).  Mask of `count` compute units spread evenly
 * over the XCDs: position i of the balanced order is slot i / num_xcds of XCD
 * i % num_xcds, and the mask takes positions [first, first + count).  The
 * ranges [0, k) and [k, num_cus) thus split the GPU into two disjoint shares
 * whose per-XCD CU counts differ by at most one.  mask: host, mask_words
 * uint32 words (bit n of word n / 32 is mask bit n), at least num_cus / 32;
 * words past the CU count are zeroed.  num_cus must be a multiple of
 * num_xcds; 1 <= count and first + count <= num_cus.
 */
opscale_status opscale_cu_mask_build(int32_t num_cus, int32_t num_xcds, int32_t interleaved, int32_t first,
                                     int32_t count, uint32_t* mask, int32_t mask_words);

/*
 * A stream restricted to the CUs set in `mask` (host, mask_words uint32
 * words, at least one bit set), at the default priority.  Kernels on it use
 * only those CUs; the library's kernels need no particular CU count.
 * Destroy it with opscale_cu_stream_destroy.
 */
opscale_status opscale_cu_stream_create(const uint32_t* mask, int32_t mask_words, hipStream_t* out);
opscale_status opscale_cu_stream_destroy(hipStream_t stream);
/* The CU mask the runtime holds for `stream` (host, mask_words words). */
opscale_status opscale_cu_stream_mask(hipStream_t stream, uint32_t* mask, int32_t mask_words);

/*
 * Placement probe: launches n_workgroups workgroups of 64 lanes on `stream`;
 * workgroup w writes out[2w] = its XCD (XCC_ID register) and out[2w + 1] =
 * the HW_ID register (CU, shader array and shader engine in bits 8..15), then
 * sleeps `spins` x 127 x 64 cycles so that the workgroups spread over every
 * CU the stream may use.  out: device, 2 * n_workgroups uint32.
 * 1 <= n_workgroups <= 65536, 0 <= spins <= 1000.  Asynchronous.
 */
opscale_status opscale_cu_probe(hipStream_t stream, uint32_t* out, int32_t n_workgroups, int32_t spins);

/* Result of opscale_corun_profile (times in microseconds). */
typedef struct {
  int32_t n_a, n_b;             /* launches of each operator in the co-run   */
  int32_t overlap_a, overlap_b; /* launches wholly inside the other's span   */
  float a_iso_us, b_iso_us;     /* T_v(b, p): median launch, each one alone  */
  float a_co_us, b_co_us;       /* T~_v(b, p): median of the overlapped ones */
  double interference_a;        /* I (Eq. 5) = a_co_us / a_iso_us            */
  double interference_b;
} opscale_corun;

/* Optional raw timestamps of opscale_corun_profile (host arrays). */
typedef struct {
  float *a_start, *a_end;  /* [max_launches]: launch i of a, from a common reference */
  float *b_start, *b_end;  /* [max_launches] */
  float *a_iso, *b_iso;    /* [iso_iters]: the isolated launch times */
} opscale_corun_trace;

/*
 * The interference factor of Eq. 5 for two operators sharing the GPU.  Each
 * runs on its own stream (sa, sb: normally CU-masked streams with disjoint
 * masks, so p is the share of each).  Both are first run `warmup` times, then
 * `iso_iters` times back to back alone on their stream, giving T_v(b, p).
 * Then both loops run at once for a window W = max(window_ms, 4 x the slower
 * of T_a, T_b): operator a launches ceil(W / T_a) times and b ceil(W / T_b)
 * times (each at least 4, at most max_launches), enqueued in the order of
 * their planned start times,
 * with device events between launches.  Launches that lie wholly inside the
 * other operator's active span give T~_v(b, p).  overlap_a or overlap_b is 0
 * (and the matching time and factor 0) when no launch qualifies.  trace may
 * be NULL.  Blocking.  1 <= iso_iters <= 4096, 4 <= max_launches <= 8192,
 * window_ms in (0, 10000].
 */
opscale_status opscale_corun_profile(const opscale_op_desc* a, hipStream_t sa, const opscale_op_desc* b,
                                     hipStream_t sb, int32_t warmup, int32_t iso_iters, float window_ms,
                                     int32_t max_launches, const opscale_corun_trace* trace, opscale_corun* out);

#ifdef __cplusplus
}
#endif
#endif /* OPSCALE_H */
