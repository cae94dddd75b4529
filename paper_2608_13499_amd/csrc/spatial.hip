// Spatial sharing of the GPU between operators: CU-masked streams, the mask
// layout over the XCDs, and a placement probe that reports where workgroups
// ran.  The paper gives each colocated operator a share of the SMs through
// its own stream (Section 2.1's SM-allocation study, Section 4.4's
// interference model); a CU mask on a HIP stream is the MI355X counterpart.
#include <hip/hip_ext.h>

#include <mutex>
#include <set>
#include <vector>

#include "opscale.h"
#include "status.h"

namespace opscale {
namespace {

constexpr int kHwRegXccId = 20;  // XCC_ID: which XCD the wave runs on (bits 3:0)
constexpr int kHwRegHwId = 4;    // HW_ID: wave, SIMD, CU, shader array, shader engine ...

// Lane 0 of each workgroup records its XCD and HW_ID, then the workgroup
// sleeps for a bounded time so that later workgroups land on other CUs.
__global__ __launch_bounds__(64) void cu_probe_kernel(uint32_t* out, int spins) {
  const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | kHwRegXccId);
  const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | kHwRegHwId);
  if (threadIdx.x == 0) {
    out[2 * (size_t)blockIdx.x] = xcc & 0xf;
    out[2 * (size_t)blockIdx.x + 1] = hw;
  }
  for (int i = 0; i < spins; ++i) __builtin_amdgcn_s_sleep(127);
}

struct Layout {
  bool known = false;
  int32_t num_cus = 0, num_xcds = 0, interleaved = 0;
};
std::mutex g_layout_mu;
Layout g_layout[64];

int popcount_words(const uint32_t* m, int32_t words) {
  int c = 0;
  for (int32_t i = 0; i < words; ++i) c += __builtin_popcount(m[i]);
  return c;
}

// Runs the probe on a stream masked to `mask` and returns the set of XCDs used.
opscale_status probe_xcds(const std::vector<uint32_t>& mask, int nwg, std::set<uint32_t>* xcds) {
  hipStream_t s = nullptr;
  hipError_t e = hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data());
  if (e != hipSuccess) return hip_fail(e, "cu_layout: hipExtStreamCreateWithCUMask");
  uint32_t* d = nullptr;
  e = hipMalloc(&d, sizeof(uint32_t) * 2 * (size_t)nwg);
  if (e != hipSuccess) {
    (void)hipStreamDestroy(s);
    return hip_fail(e, "cu_layout: hipMalloc");
  }
  std::vector<uint32_t> h(2 * (size_t)nwg);
  hipLaunchKernelGGL(cu_probe_kernel, dim3((unsigned)nwg), dim3(64), 0, s, d, 4);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpyAsync(h.data(), d, h.size() * sizeof(uint32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  (void)hipFree(d);
  (void)hipStreamDestroy(s);
  if (e != hipSuccess) return hip_fail(e, "cu_layout: probe");
  for (int w = 0; w < nwg; ++w) xcds->insert(h[2 * (size_t)w]);
  return OPSCALE_OK;
}

}  // namespace
}  // namespace opscale

using opscale::fail;
using opscale::hip_fail;

extern "C" {

opscale_status opscale_cu_mask_build(int32_t num_cus, int32_t num_xcds, int32_t interleaved, int32_t first,
                                     int32_t count, uint32_t* mask, int32_t mask_words) {
  if (!mask) return fail(OPSCALE_ERR_INVALID_ARG, "cu_mask_build: null mask");
  if (num_cus < 1 || num_xcds < 1 || num_cus % num_xcds != 0)
    return fail(OPSCALE_ERR_INVALID_ARG, "cu_mask_build: num_cus (%d) must be a positive multiple of num_xcds (%d)",
                num_cus, num_xcds);
  if (mask_words < (num_cus + 31) / 32)
    return fail(OPSCALE_ERR_INVALID_ARG, "cu_mask_build: %d words cannot hold %d CUs", mask_words, num_cus);
  if (count < 1 || first < 0 || (int64_t)first + count > num_cus)
    return fail(OPSCALE_ERR_INVALID_ARG, "cu_mask_build: positions [%d, %d + %d) outside [0, %d)", first, first,
                count, num_cus);
  const int32_t per_xcd = num_cus / num_xcds;
  for (int32_t w = 0; w < mask_words; ++w) mask[w] = 0u;
  for (int32_t i = first; i < first + count; ++i) {
    const int32_t x = i % num_xcds, slot = i / num_xcds;
    const int32_t bit = interleaved ? slot * num_xcds + x : x * per_xcd + slot;
    mask[bit >> 5] |= 1u << (bit & 31);
  }
  return OPSCALE_OK;
}

opscale_status opscale_cu_layout(int32_t* num_cus, int32_t* num_xcds, int32_t* interleaved) {
  if (!num_cus || !num_xcds || !interleaved) return fail(OPSCALE_ERR_INVALID_ARG, "cu_layout: null output");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "cu_layout: hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(OPSCALE_ERR_UNSUPPORTED, "cu_layout: device %d", dev);
  std::lock_guard<std::mutex> lock(opscale::g_layout_mu);
  opscale::Layout& L = opscale::g_layout[dev];
  if (!L.known) {
    int cus = 0, xcds = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return hip_fail(e, "cu_layout: CU count");
    if ((e = hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev)) != hipSuccess)
      return hip_fail(e, "cu_layout: XCC count");
    if (cus < 1 || xcds < 1 || cus % xcds != 0)
      return fail(OPSCALE_ERR_UNSUPPORTED, "cu_layout: %d CUs over %d XCDs", cus, xcds);
    int inter = 1;
    if (xcds > 1) {
      // the first cus / xcds mask bits: all on XCD 0 if the mask is blocked by
      // XCD, one CU set per XCD if it is interleaved
      std::vector<uint32_t> m((size_t)(cus + 31) / 32, 0u);
      for (int b = 0; b < cus / xcds; ++b) m[(size_t)b >> 5] |= 1u << (b & 31);
      std::set<uint32_t> used;
      const opscale_status st = opscale::probe_xcds(m, 4 * cus, &used);
      if (st != OPSCALE_OK) return st;
      if ((int)used.size() == xcds) inter = 1;
      else if (used.size() == 1) inter = 0;
      else
        return fail(OPSCALE_ERR_UNSUPPORTED, "cu_layout: the first %d mask bits ran on %zu of %d XCDs", cus / xcds,
                    used.size(), xcds);
    }
    L.num_cus = cus;
    L.num_xcds = xcds;
    L.interleaved = inter;
    L.known = true;
  }
  *num_cus = L.num_cus;
  *num_xcds = L.num_xcds;
  *interleaved = L.interleaved;
  return OPSCALE_OK;
}

opscale_status opscale_cu_stream_create(const uint32_t* mask, int32_t mask_words, hipStream_t* out) {
  if (!mask || !out || mask_words < 1) return fail(OPSCALE_ERR_INVALID_ARG, "cu_stream_create: null mask or out");
  if (opscale::popcount_words(mask, mask_words) == 0)
    return fail(OPSCALE_ERR_INVALID_ARG, "cu_stream_create: the mask selects no CU");
  const hipError_t e = hipExtStreamCreateWithCUMask(out, (uint32_t)mask_words, mask);
  if (e != hipSuccess) return hip_fail(e, "hipExtStreamCreateWithCUMask");
  return OPSCALE_OK;
}

opscale_status opscale_cu_stream_destroy(hipStream_t stream) {
  if (!stream) return fail(OPSCALE_ERR_INVALID_ARG, "cu_stream_destroy: null stream");
  const hipError_t e = hipStreamDestroy(stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamDestroy");
  return OPSCALE_OK;
}

opscale_status opscale_cu_stream_mask(hipStream_t stream, uint32_t* mask, int32_t mask_words) {
  if (!mask || mask_words < 1) return fail(OPSCALE_ERR_INVALID_ARG, "cu_stream_mask: null mask");
  const hipError_t e = hipExtStreamGetCUMask(stream, (uint32_t)mask_words, mask);
  if (e != hipSuccess) return hip_fail(e, "hipExtStreamGetCUMask");
  return OPSCALE_OK;
}

opscale_status opscale_cu_probe(hipStream_t stream, uint32_t* out, int32_t n_workgroups, int32_t spins) {
  if (!out) return fail(OPSCALE_ERR_INVALID_ARG, "cu_probe: null out");
  if (n_workgroups < 1 || n_workgroups > 65536)
    return fail(OPSCALE_ERR_INVALID_ARG, "cu_probe: n_workgroups %d outside [1, 65536]", n_workgroups);
  if (spins < 0 || spins > 1000) return fail(OPSCALE_ERR_INVALID_ARG, "cu_probe: spins %d outside [0, 1000]", spins);
  hipLaunchKernelGGL(opscale::cu_probe_kernel, dim3((unsigned)n_workgroups), dim3(64), 0, stream, out, spins);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "cu_probe launch");
  return OPSCALE_OK;
}

}  // extern "C"
