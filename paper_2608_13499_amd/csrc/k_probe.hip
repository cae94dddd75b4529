// Peak probes: what the matrix cores and HBM deliver on this GPU, measured,
// to report the operators against beside the published peaks (the paper
// characterizes each operator by how much of the GPU it uses, Section 2.1).
//
// MFMA: every wave runs 8 independent chains of v_mfma_f32_16x16x32_bf16 on
// register operands (non-zero bf16 values, so the power draw is that of real
// data), 4 waves per SIMD.  HBM: a grid-stride stream of 16-byte nontemporal
// loads (read probe) or loads and stores (copy probe) over a caller buffer.
#include <hip/hip_runtime.h>

#include "common.h"
#include "opscale.h"
#include "status.h"

namespace opscale {
namespace {

constexpr int kProbeChains = 8;

// 512-thread workgroups cap a wave at 128 registers, which keeps the
// accumulators in VGPRs updated in place (with the larger budget of smaller
// workgroups the compiler puts them in AGPRs and rotates them every trip).
__global__ __launch_bounds__(512) void mfma_peak_kernel(int64_t iters) {
  const uint32_t t = threadIdx.x + blockIdx.x * 512u;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.5f + 0.001f * (float)((t * 7u + i) & 63u));
    b[i] = (__bf16)(0.25f - 0.002f * (float)((t * 13u + i) & 31u));
  }
  f32x4 acc[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // iters: a multiple of 4, at most 2^24 (set by the host); 4 rounds of the chains per trip.
  const int32_t trips = (int32_t)iters;
  for (int32_t it = 0; it < trips; it += 4) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int j = 0; j < kProbeChains; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  asm volatile("" :: "v"(s));  // consumes the chains, so none is dropped
}

// 2 independent 16-byte nontemporal loads per lane per step, 3 workgroups
// of 256 per CU: the launch shape that streamed fastest among 1-4 loads per
// lane and 0.5-8 workgroups per CU (more loads in flight than this lowers
// the rate).  The read probe folds what it reads into an XOR that an empty
// asm statement consumes, so it writes nothing.
constexpr int kHbmWgPerCu = 3;

__global__ __launch_bounds__(256) void hbm_read_kernel(const u32x4* __restrict__ src, int64_t nvec) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  u32x4 x = {0u, 0u, 0u, 0u};
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + stride < nvec; i += 2 * stride) {
    const u32x4 v0 = __builtin_nontemporal_load(src + i), v1 = __builtin_nontemporal_load(src + i + stride);
    x ^= v0 ^ v1;
  }
  if (i < nvec) x ^= __builtin_nontemporal_load(src + i);
  const uint32_t r = x[0] ^ x[1] ^ x[2] ^ x[3];
  asm volatile("" :: "v"(r));
}

__global__ __launch_bounds__(256) void hbm_copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                       int64_t nvec) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + stride < nvec; i += 2 * stride) {
    const u32x4 v0 = __builtin_nontemporal_load(src + i), v1 = __builtin_nontemporal_load(src + i + stride);
    __builtin_nontemporal_store(v0, dst + i);
    __builtin_nontemporal_store(v1, dst + i + stride);
  }
  if (i < nvec) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// Times reps launches of `launch` on s with a pair of events (after one
// untimed launch); returns the mean microseconds per launch.
template <class F>
opscale_status time_reps(hipStream_t s, int32_t reps, const char* what, F&& launch, double* us) {
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) e = launch();
  if (e == hipSuccess) e = hipEventRecord(a, s);
  for (int32_t r = 0; r < reps && e == hipSuccess; ++r) e = launch();
  if (e == hipSuccess) e = hipEventRecord(b, s);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (e != hipSuccess) return hip_fail(e, what);
  *us = (double)ms * 1000.0 / reps;
  return OPSCALE_OK;
}

}  // namespace
}  // namespace opscale

using opscale::fail;

extern "C" {

opscale_status opscale_probe_mfma(int64_t iters, int32_t reps, hipStream_t stream, double* tflops) {
  if (!tflops) return fail(OPSCALE_ERR_INVALID_ARG, "probe_mfma: null result pointer");
  if (iters < 1 || iters > ((int64_t)1 << 24) || reps < 1 || reps > 1000)
    return fail(OPSCALE_ERR_INVALID_ARG, "probe_mfma: iters=%lld (1..2^24) reps=%d (1..1000)", (long long)iters, reps);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return opscale::hip_fail(e, "probe_mfma: device query");
  const int64_t iters4 = (iters + 3) / 4 * 4;  // the kernel runs the chains in groups of 4
  const unsigned blocks = (unsigned)cus * 2;  // 2 workgroups of 8 waves: 4 waves per SIMD
  double us = 0.0;
  const opscale_status st = opscale::time_reps(stream, reps, "probe_mfma launch", [&] {
    hipLaunchKernelGGL(opscale::mfma_peak_kernel, dim3(blocks), dim3(512), 0, stream, iters4);
    return hipGetLastError();
  }, &us);
  if (st != OPSCALE_OK) return st;
  const double flops = (double)blocks * 8 * (double)iters4 * opscale::kProbeChains * (2.0 * 16 * 16 * 32);
  *tflops = flops / (us * 1e-6) / 1e12;
  return OPSCALE_OK;
}

opscale_status opscale_probe_hbm(const void* src, void* dst, size_t bytes, int32_t reps, hipStream_t stream,
                                 double* gbps) {
  if (!gbps || !src) return fail(OPSCALE_ERR_INVALID_ARG, "probe_hbm: null pointer");
  if (bytes < 16 || bytes % 16 || reps < 1 || reps > 1000)
    return fail(OPSCALE_ERR_INVALID_ARG, "probe_hbm: bytes=%zu (a multiple of 16) reps=%d (1..1000)", bytes, reps);
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15)
    return fail(OPSCALE_ERR_INVALID_ARG, "probe_hbm: buffers must be 16-byte aligned");
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (dst && s0 < d0 + bytes && d0 < s0 + bytes)
    return fail(OPSCALE_ERR_INVALID_ARG, "probe_hbm: dst must not overlap src");
  const int64_t nvec = (int64_t)(bytes / 16);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return opscale::hip_fail(e, "probe_hbm: device query");
  const unsigned blocks = (unsigned)cus * opscale::kHbmWgPerCu;
  double us = 0.0;
  const auto* s16 = static_cast<const opscale::u32x4*>(src);
  auto* d16 = static_cast<opscale::u32x4*>(dst);
  const opscale_status st = opscale::time_reps(stream, reps, "probe_hbm launch", [&] {
    if (dst)
      hipLaunchKernelGGL(opscale::hbm_copy_kernel, dim3(blocks), dim3(256), 0, stream, s16, d16, nvec);
    else
      hipLaunchKernelGGL(opscale::hbm_read_kernel, dim3(blocks), dim3(256), 0, stream, s16, nvec);
    return hipGetLastError();
  }, &us);
  if (st != OPSCALE_OK) return st;
  *gbps = (double)bytes * (dst ? 2.0 : 1.0) / (us * 1e-6) / 1e9;
  return OPSCALE_OK;
}

}  // extern "C"
