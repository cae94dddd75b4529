/* Host-only driver for the AddressSanitizer check of the C ABI's validation
 * layer: every entry point is called with arguments it must reject (null or
 * misaligned pointers, overlapping tensors, bad sizes, too-small workspaces,
 * unknown knobs) and the documented status code is checked.  Every call
 * returns before anything reaches a device, so no GPU is needed.  Exit status:
 * the number of mismatches (0: all as documented). */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "opscale.h"

static int g_bad = 0;

#define EXPECT(call, want)                                                                       \
  do {                                                                                           \
    const int got_ = (int)(call);                                                                \
    if (got_ != (int)(want)) {                                                                   \
      fprintf(stderr, "line %d: %s returned %d, expected %d (%s)\n", __LINE__, #call, got_,      \
              (int)(want), opscale_last_error());                                                \
      ++g_bad;                                                                                   \
    }                                                                                            \
  } while (0)

/* Fake device addresses: 16-byte aligned, far apart, never dereferenced. */
#define A(i) ((void*)((uintptr_t)(i) << 34))

int main(void) {
  const opscale_status INV = OPSCALE_ERR_INVALID_ARG, UNS = OPSCALE_ERR_UNSUPPORTED, WS = OPSCALE_ERR_WORKSPACE;
  if (!strstr(opscale_version(), "gfx950")) ++g_bad;
  if (strcmp(opscale_status_string(OPSCALE_ERR_WORKSPACE), "workspace too small") != 0) ++g_bad;

  /* RMS Norm */
  EXPECT(opscale_rmsnorm(NULL, NULL, NULL, 4, 4096, 1e-5f, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_rmsnorm(A(1), A(2), A(3), 4, 4095, 1e-5f, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_rmsnorm((char*)A(1) + 2, A(2), A(3), 4, 4096, 1e-5f, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_rmsnorm(A(1), A(2), (char*)A(1) + 16, 4, 4096, 1e-5f, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_rmsnorm(A(1), A(2), A(3), 4, 4096, -1.f, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_rmsnorm(A(1), A(2), A(3), 4, 4096, 1e-5f, (opscale_dtype)7, 0, NULL), INV);
  EXPECT(opscale_rmsnorm(NULL, NULL, NULL, 0, 4096, 1e-5f, OPSCALE_BF16, 0, NULL), OPSCALE_OK);

  /* linear, its workspace and the tuning hook */
  EXPECT(opscale_linear(A(1), A(2), NULL, A(3), 8, 256, 100, OPSCALE_BF16, NULL, 0, 0, NULL), INV);
  EXPECT(opscale_linear(A(1), A(2), NULL, A(1), 8, 256, 64, OPSCALE_BF16, NULL, 0, 0, NULL), INV);
  EXPECT(opscale_linear(A(1), NULL, NULL, A(3), 8, 256, 64, OPSCALE_BF16, NULL, 0, 0, NULL), INV);
  EXPECT(opscale_linear(A(1), A(2), (char*)A(4) + 4, A(3), 8, 256, 64, OPSCALE_BF16, NULL, 0, 0, NULL), INV);
  const size_t need = opscale_linear_workspace_size(100, 4096, 4096, OPSCALE_BF16);
  if (need != (size_t)8 * 100 * 4096 * 4) ++g_bad;
  EXPECT(opscale_linear(A(1), A(2), NULL, A(3), 100, 4096, 4096, OPSCALE_BF16, A(4), need - 1, 0, NULL), WS);
  EXPECT(opscale_linear(A(1), A(2), NULL, A(3), 100, 4096, 4096, OPSCALE_BF16, A(3), need, 0, NULL), INV);
  EXPECT(opscale_set_tuning((opscale_tune)99, 0), INV);
  EXPECT(opscale_set_tuning(OPSCALE_TUNE_GEMM_TILE, 4), INV);
  EXPECT(opscale_set_tuning(OPSCALE_TUNE_GEMM_SPLITK, 0), OPSCALE_OK);
  if (opscale_linear_workspace_size(100, 4096, 4096, OPSCALE_BF16) != 0) ++g_bad;
  EXPECT(opscale_set_tuning(OPSCALE_TUNE_GEMM_SPLITK, -1), OPSCALE_OK);

  /* SwiGLU */
  EXPECT(opscale_swiglu(A(1), A(1), 8, 256, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_swiglu(A(1), A(2), 8, 3, OPSCALE_F32, 0, NULL), INV);

  /* prefill attention */
  EXPECT(opscale_attn_prefill(A(1), A(2), A(3), 48 * 128, 48 * 128, A(4), (const int32_t*)A(5), 2, 100, 64, 32, 5,
                              128, 0.08f, 1, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_attn_prefill(A(1), A(2), A(3), 48 * 128, 48 * 128, A(4), (const int32_t*)A(5), 2, 100, 64, 32, 8,
                              96, 0.08f, 1, OPSCALE_BF16, 0, NULL), UNS);
  EXPECT(opscale_attn_prefill(A(1), A(2), A(3), 48 * 128, 48 * 128, A(4), NULL, 2, 100, 64, 32, 8, 128, 0.08f, 1,
                              OPSCALE_BF16, 0, NULL), INV);

  /* decode attention: workspace and the allocation-free entry point's limit */
  const size_t dneed = opscale_attn_decode_workspace_size(256, 32, 128, 8192);
  EXPECT(opscale_attn_decode(A(1), 32 * 128, A(2), A(3), (const int32_t*)A(4), (const int32_t*)A(5), A(6), 256, 32,
                             8, 128, 16, 512, 70000, 8192, 0.08f, OPSCALE_BF16, A(7), dneed - 1, 0, NULL), WS);
  EXPECT(opscale_attn_decode(A(1), 32 * 128, A(2), A(3), (const int32_t*)A(4), (const int32_t*)A(5), A(6), 256, 32,
                             8, 96, 16, 512, 70000, 8192, 0.08f, OPSCALE_BF16, A(7), dneed, 0, NULL), UNS);
  if (opscale_attn_decode_noalloc_max_bytes() != ((size_t)64 << 20)) ++g_bad;

  /* RoPE, cache write, residual norm */
  EXPECT(opscale_rope(A(1), A(2), 48 * 128, 48 * 128, NULL, 10, 32, 8, 128, 500000.0, OPSCALE_BF16, 0, NULL), INV);
  EXPECT(opscale_reshape_and_cache(A(1), A(2), 48 * 128, A(3), A(4), NULL, 10, 8, 128, 16, 1024, OPSCALE_BF16, 0,
                                   NULL), INV);
  EXPECT(opscale_add_rmsnorm(A(1), A(2), A(3), A(2), 4, 4096, 1e-5f, OPSCALE_BF16, 0, NULL), INV);

  /* mixture of experts */
  const size_t mneed = opscale_fused_moe_workspace_size(64, 128, 256, 8, 2);
  EXPECT(opscale_fused_moe(A(1), A(2), A(3), (const int32_t*)A(4), (const float*)A(5), A(6), 64, 128, 256, 8, 2,
                           OPSCALE_BF16, A(7), mneed - 1, 0, NULL), WS);
  EXPECT(opscale_moe_topk((const float*)A(1), (int32_t*)A(2), (float*)A(3), 10, 8, 9, 1, 0, NULL), INV);

  /* the profile descriptor */
  opscale_op_desc d;
  memset(&d, 0, sizeof d);
  d.op = (opscale_op)42;
  d.dt = OPSCALE_BF16;
  opscale_profile prof;
  EXPECT(opscale_op_profile(&d, 1, 1, NULL, 0, 0, &prof), INV);
  EXPECT(opscale_op_profile(NULL, 1, 1, NULL, 0, 0, &prof), INV);

  /* CU masks */
  uint32_t words[8];
  EXPECT(opscale_cu_mask_build(256, 8, 1, 250, 10, words, 8), INV);

  if (g_bad) fprintf(stderr, "%d mismatches\n", g_bad);
  return g_bad;
}
