// Bandwidth-bound operators: RMS Norm and the fused SiLU-multiply (SwiGLU).
//
// Both stream their operands once from HBM with 16-byte loads and stores per
// lane, keep the math in fp32 and round once at the output.
#include "common.h"
#include "launch.h"

namespace opscale {

// ------------------------------------------------------------- RMS Norm ----
// One wave per row.  VPL = 16-byte vectors per lane held in registers (a row of
// up to VPL*64*16 bytes is read once); VPL == 0 selects the streaming variant
// for longer rows, which reads the row a second time (from L2) to normalize.
template <bool BF16, int VPL>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const void* x, const void* __restrict__ w,
                                                      void* y, int64_t M,
                                                      int H, float eps) {
  constexpr int EPV = BF16 ? 8 : 4;  // elements per 16-byte vector
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int nvec = H / EPV;
  const u32x4* xr = reinterpret_cast<const u32x4*>(static_cast<const char*>(x) + row * (int64_t)H * (BF16 ? 2 : 4));
  u32x4* yr = reinterpret_cast<u32x4*>(static_cast<char*>(y) + row * (int64_t)H * (BF16 ? 2 : 4));
  const u32x4* wr = reinterpret_cast<const u32x4*>(w);

  auto sq = [](const u32x4& v) {
    float s = 0.f;
    if constexpr (BF16) {
      const uint32_t a[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float lo = bf_lo(a[i]), hi = bf_hi(a[i]);
        s = fmaf(lo, lo, s);
        s = fmaf(hi, hi, s);
      }
    } else {
      const float a[4] = {__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                          __uint_as_float(v[3])};
#pragma unroll
      for (int i = 0; i < 4; ++i) s = fmaf(a[i], a[i], s);
    }
    return s;
  };
  auto scale = [](const u32x4& v, const u32x4& g, float r) {
    u32x4 o;
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        o[i] = pack_bf2(bf_lo(v[i]) * r * bf_lo(g[i]), bf_hi(v[i]) * r * bf_hi(g[i]));
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        o[i] = __float_as_uint(__uint_as_float(v[i]) * r * __uint_as_float(g[i]));
    }
    return o;
  };

  float ss = 0.f;
  if constexpr (VPL > 0) {
    // the row and the weight are requested together, so the weight (an L2
    // hit) costs no round trip after the reduction.  Plain (cached) loads and
    // stores: measured 1-2 us faster on an 8871 x 4096 row block than the
    // nontemporal forms, and faster than a device copy of the same bytes.
    u32x4 v[VPL], g[VPL];
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int idx = lane + i * 64;
      v[i] = idx < nvec ? xr[idx] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int idx = lane + i * 64;
      g[i] = idx < nvec ? wr[idx] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < VPL; ++i) ss += sq(v[i]);
    ss = wave_sum_f(ss);
    const float r = rsqrtf(ss / (float)H + eps);
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int idx = lane + i * 64;
      if (idx < nvec) yr[idx] = scale(v[i], g[i], r);
    }
  } else {
    for (int idx = lane; idx < nvec; idx += 64) ss += sq(xr[idx]);
    ss = wave_sum(ss);
    const float r = rsqrtf(ss / (float)H + eps);
    for (int idx = lane; idx < nvec; idx += 64) yr[idx] = scale(xr[idx], wr[idx], r);
  }
}

template <bool BF16>
static hipError_t rmsnorm_dispatch(const void* x, const void* w, void* y, int64_t M, int64_t H,
                                   float eps, hipStream_t s) {
  const int epv = BF16 ? 8 : 4;
  const int64_t nvec = H / epv;
  const int vpl = (int)((nvec + 63) / 64);
  const dim3 grid((unsigned)((M + 3) / 4)), block(256);
  const int h = (int)H;
#define OPS_RMS(V) hipLaunchKernelGGL((rmsnorm_kernel<BF16, V>), grid, block, 0, s, x, w, y, M, h, eps)
  if (vpl <= 1) OPS_RMS(1);
  else if (vpl <= 2) OPS_RMS(2);
  else if (vpl <= 4) OPS_RMS(4);
  else if (vpl <= 8) OPS_RMS(8);
  else if (vpl <= 16) OPS_RMS(16);
  else OPS_RMS(0);
#undef OPS_RMS
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const void* x, const void* w, void* y, int64_t M, int64_t H, float eps,
                          bool bf16, hipStream_t s) {
  return bf16 ? rmsnorm_dispatch<true>(x, w, y, M, H, eps, s)
              : rmsnorm_dispatch<false>(x, w, y, M, H, eps, s);
}

// --------------------------------------------------------------- SwiGLU ----
// grid.x covers one row's 16-byte output vectors (256 threads x VPT vectors
// each), grid.y strides over rows.
template <bool BF16, int VPT>
__global__ __launch_bounds__(256) void swiglu_kernel(const void* __restrict__ gu, void* __restrict__ out,
                                                     int64_t M, int64_t F) {
  constexpr int EPV = BF16 ? 8 : 4;
  constexpr int ES = BF16 ? 2 : 4;
  const int64_t nvec = F / EPV;
  for (int64_t row = blockIdx.y; row < M; row += gridDim.y) {
    const u32x4* g = reinterpret_cast<const u32x4*>(static_cast<const char*>(gu) + row * 2 * F * ES);
    const u32x4* u = reinterpret_cast<const u32x4*>(static_cast<const char*>(gu) + (row * 2 * F + F) * ES);
    u32x4* o = reinterpret_cast<u32x4*>(static_cast<char*>(out) + row * F * ES);
    u32x4 gv[VPT], uv[VPT];
    const int64_t base = (int64_t)blockIdx.x * 256 * VPT + threadIdx.x;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int64_t idx = base + i * 256;
      if (idx < nvec) {
        gv[i] = __builtin_nontemporal_load(g + idx);
        uv[i] = __builtin_nontemporal_load(u + idx);
      }
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int64_t idx = base + i * 256;
      if (idx >= nvec) continue;
      const u32x4 ga = gv[i], ua = uv[i];
      u32x4 r;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if constexpr (BF16) {
          const float g0 = bf_lo(ga[e]), g1 = bf_hi(ga[e]);
          const float s0 = g0 / (1.f + __expf(-g0)), s1 = g1 / (1.f + __expf(-g1));
          r[e] = pack_bf2(s0 * bf_lo(ua[e]), s1 * bf_hi(ua[e]));
        } else {
          const float g0 = __uint_as_float(ga[e]);
          r[e] = __float_as_uint(g0 / (1.f + expf(-g0)) * __uint_as_float(ua[e]));
        }
      }
      __builtin_nontemporal_store(r, o + idx);
    }
  }
}

hipError_t launch_swiglu(const void* gu, void* out, int64_t M, int64_t F, bool bf16, hipStream_t s) {
  constexpr int VPT = 2;
  const int64_t nvec = F / (bf16 ? 8 : 4);
  const unsigned gx = (unsigned)((nvec + 256 * VPT - 1) / (256 * VPT));
  const unsigned gy = (unsigned)(M < 65535 ? M : 65535);
  if (bf16)
    hipLaunchKernelGGL((swiglu_kernel<true, VPT>), dim3(gx, gy), dim3(256), 0, s, gu, out, M, F);
  else
    hipLaunchKernelGGL((swiglu_kernel<false, VPT>), dim3(gx, gy), dim3(256), 0, s, gu, out, M, F);
  return hipGetLastError();
}

// ---------------------------------------------------------------- flush ----
// Reads every byte of buf, so the caches then hold clean lines of buf and
// nothing of the timed operator's operands.  (A writing flush would leave the
// last-level cache full of dirty lines, and the next kernel would pay for
// their write-back.)  The XOR of the data is stored only if it equals `tag`,
// which keeps the loads alive and practically never happens.
__global__ __launch_bounds__(256) void flush_kernel(u32x4* buf, size_t nvec, uint32_t tag) {
  uint32_t h = 0;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < nvec; i += (size_t)gridDim.x * 256) {
    const u32x4 v = buf[i];  // a plain load: it allocates in L2 and the MALL
    h ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  const size_t me = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (h == tag && me < nvec) buf[me][0] = h;
}

hipError_t launch_flush(void* buf, size_t bytes, hipStream_t s) {
  const size_t nvec = bytes / 16;
  if (nvec == 0) return hipSuccess;
  hipLaunchKernelGGL(flush_kernel, dim3(2048), dim3(256), 0, s, static_cast<u32x4*>(buf), nvec,
                     0x5a5a5a5au);
  return hipGetLastError();
}

}  // namespace opscale
