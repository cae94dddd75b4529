// Stream-ordered device scratch for kernels that need temporary buffers the
// caller does not pass (the split-K partial tiles of the linear layer).  Each
// device gets one memory pool owned by the library, with no release
// threshold, so memory freed at the end of a call is reused by the next one
// instead of going back to the driver; allocation and release are ordered on
// the caller's stream, so calls on different streams never share a buffer.
#include <cstdint>
#include <mutex>

#include "launch.h"

namespace opscale {
namespace {
std::mutex g_pool_mu;
hipMemPool_t g_pool[64];
}  // namespace

static hipError_t device_pool(hipMemPool_t* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  if (!g_pool[dev]) {
    hipMemPoolProps props = {};
    props.allocType = hipMemAllocationTypePinned;
    props.handleTypes = hipMemHandleTypeNone;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool = nullptr;
    if ((e = hipMemPoolCreate(&pool, &props)) != hipSuccess) return e;
    uint64_t keep = UINT64_MAX;
    if ((e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep)) != hipSuccess) {
      (void)hipMemPoolDestroy(pool);
      return e;
    }
    g_pool[dev] = pool;
  }
  *out = g_pool[dev];
  return hipSuccess;
}

hipError_t scratch_alloc(size_t bytes, hipStream_t s, void** p) {
  hipMemPool_t pool = nullptr;
  const hipError_t e = device_pool(&pool);
  if (e != hipSuccess) return e;
  return hipMallocFromPoolAsync(p, bytes, pool, s);
}

hipError_t scratch_free(void* p, hipStream_t s) { return hipFreeAsync(p, s); }

}  // namespace opscale
