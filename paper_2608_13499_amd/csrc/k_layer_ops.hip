// The operators around attention in a decoder layer: rotary embedding of q
// and k, the paged KV-cache write, and the residual add fused into RMS Norm.
// All three are bandwidth-bound; each moves its operands once with 8- or
// 16-byte accesses per lane and computes in fp32 (the RoPE angle in fp64).
#include <cmath>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr double kTwoPi = 6.283185307179586476925286766559;
}  // namespace

// ------------------------------------------------------------------ RoPE ----
// One workgroup per token.  A thread owns 4 consecutive rotation pairs
// (i .. i + 3, partners i + D/2 .. i + D/2 + 3) of one head, q heads first
// then k heads.  The angle p * theta^(-2i/D) is formed in fp64 and reduced to
// [-pi, pi] there, so the fp32 sine and cosine see an argument accurate to
// ~1e-7 rad at any position.
template <bool BF16, int D>
__global__ __launch_bounds__(256) void rope_kernel(void* q, void* k, int64_t q_stride, int64_t k_stride,
                                                   const int32_t* __restrict__ pos, int Hq, int Hkv,
                                                   double log2_theta) {
  constexpr int HALF = D / 2, QUADS = HALF / 4;
  __shared__ double inv_freq[HALF];
  for (int i = threadIdx.x; i < HALF; i += 256) inv_freq[i] = exp2(-(2.0 * i / D) * log2_theta);
  __syncthreads();
  const int64_t t = blockIdx.x;
  const double p = (double)pos[t];
  for (int idx = threadIdx.x; idx < (Hq + Hkv) * QUADS; idx += 256) {
    const int head = idx / QUADS, quad = idx % QUADS;
    const int64_t row = head < Hq ? t * q_stride + (int64_t)head * D : t * k_stride + (int64_t)(head - Hq) * D;
    void* base = head < Hq ? q : k;
    float a[4], b[4];
    if constexpr (BF16) {
      __bf16* e = static_cast<__bf16*>(base) + row + 4 * quad;
      const u32x2 lo = *reinterpret_cast<const u32x2*>(e);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(e + HALF);
      a[0] = bf_lo(lo[0]), a[1] = bf_hi(lo[0]), a[2] = bf_lo(lo[1]), a[3] = bf_hi(lo[1]);
      b[0] = bf_lo(hi[0]), b[1] = bf_hi(hi[0]), b[2] = bf_lo(hi[1]), b[3] = bf_hi(hi[1]);
    } else {
      float* e = static_cast<float*>(base) + row + 4 * quad;
      const u32x4 lo = *reinterpret_cast<const u32x4*>(e);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(e + HALF);
#pragma unroll
      for (int j = 0; j < 4; ++j) a[j] = __uint_as_float(lo[j]), b[j] = __uint_as_float(hi[j]);
    }
    float ra[4], rb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double ang = p * inv_freq[4 * quad + j];
      const float r = (float)(ang - kTwoPi * rint(ang * (1.0 / kTwoPi)));
      float sn, cs;
      sincosf(r, &sn, &cs);
      ra[j] = a[j] * cs - b[j] * sn;
      rb[j] = b[j] * cs + a[j] * sn;
    }
    if constexpr (BF16) {
      __bf16* e = static_cast<__bf16*>(base) + row + 4 * quad;
      *reinterpret_cast<u32x2*>(e) = u32x2{pack_bf2(ra[0], ra[1]), pack_bf2(ra[2], ra[3])};
      *reinterpret_cast<u32x2*>(e + HALF) = u32x2{pack_bf2(rb[0], rb[1]), pack_bf2(rb[2], rb[3])};
    } else {
      float* e = static_cast<float*>(base) + row + 4 * quad;
      *reinterpret_cast<u32x4*>(e) =
          u32x4{__float_as_uint(ra[0]), __float_as_uint(ra[1]), __float_as_uint(ra[2]), __float_as_uint(ra[3])};
      *reinterpret_cast<u32x4*>(e + HALF) =
          u32x4{__float_as_uint(rb[0]), __float_as_uint(rb[1]), __float_as_uint(rb[2]), __float_as_uint(rb[3])};
    }
  }
}

hipError_t launch_rope(void* q, void* k, int64_t q_stride, int64_t k_stride, const int32_t* pos, int64_t T,
                       int32_t Hq, int32_t Hkv, int32_t D, double theta, bool bf16, hipStream_t s) {
  const double l2 = std::log2(theta);
  const dim3 grid((unsigned)T), block(256);
#define OPS_ROPE(B, DD) \
  hipLaunchKernelGGL((rope_kernel<B, DD>), grid, block, 0, s, q, k, q_stride, k_stride, pos, Hq, Hkv, l2)
  if (bf16) {
    if (D == 128) OPS_ROPE(true, 128);
    else OPS_ROPE(true, 64);
  } else {
    if (D == 128) OPS_ROPE(false, 128);
    else OPS_ROPE(false, 64);
  }
#undef OPS_ROPE
  return hipGetLastError();
}

// ------------------------------------------------------- KV cache write ----
// The rows to copy are a list of 16-byte chunks: token t owns chunks
// [t * 2 * row_chunks, (t + 1) * 2 * row_chunks), its K row first, then its V
// row, each copied to cache row `slot` (the cache [num_blocks, block_size,
// Hkv, D] is an array of such rows).  A workgroup takes kChunksPerWg
// consecutive chunks, a thread kCwPerThread of them 256 apart: every load (the
// row chunks and their tokens' slots) is issued before the first store.
// Tokens whose slot is outside [0, num_slots) are skipped.
constexpr int kCwPerThread = 4;
constexpr int kChunksPerWg = 256 * kCwPerThread;
__global__ __launch_bounds__(256) void cache_write_kernel(const char* __restrict__ k, const char* __restrict__ v,
                                                         int64_t kv_stride_bytes, char* kc, char* vc,
                                                         const int32_t* __restrict__ slots, int row_chunks,
                                                         int64_t T, int64_t num_slots) {
  const int64_t total = T * 2 * row_chunks;
  for (int64_t blk = blockIdx.x; blk * kChunksPerWg < total; blk += gridDim.x) {
  const int64_t q0 = blk * kChunksPerWg + threadIdx.x;
  u32x4 val[kCwPerThread];
  int64_t slot[kCwPerThread];
#pragma unroll
  for (int i = 0; i < kCwPerThread; ++i) {
    const int64_t q = min(q0 + i * 256, total - 1);  // clamped: the stores below check q
    const int64_t t = q / (2 * row_chunks);
    const int c = (int)(q - t * 2 * row_chunks);
    const bool isv = c >= row_chunks;
    val[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>((isv ? v : k) + t * kv_stride_bytes) +
                                        (isv ? c - row_chunks : c));
    slot[i] = slots[t];
  }
#pragma unroll
  for (int i = 0; i < kCwPerThread; ++i) {
    const int64_t q = q0 + i * 256;
    if (q >= total || slot[i] < 0 || slot[i] >= num_slots) continue;
    const int64_t t = q / (2 * row_chunks);
    const int c = (int)(q - t * 2 * row_chunks);
    const bool isv = c >= row_chunks;
    *(reinterpret_cast<u32x4*>((isv ? vc : kc) + slot[i] * (int64_t)row_chunks * 16) + (isv ? c - row_chunks : c)) =
        val[i];
  }
  }  // block stride
}

hipError_t launch_cache_write(const void* k, const void* v, int64_t kv_stride, void* kc, void* vc,
                              const int32_t* slots, int64_t T, int32_t Hkv, int32_t D, int64_t num_slots,
                              bool bf16, hipStream_t s) {
  const int es = bf16 ? 2 : 4;
  const int row_chunks = (int)((int64_t)Hkv * D * es / 16);
  const int64_t total = T * 2 * row_chunks;
  const int64_t blocks = std::min<int64_t>((total + kChunksPerWg - 1) / kChunksPerWg, 1 << 20);
  hipLaunchKernelGGL(cache_write_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     static_cast<const char*>(k), static_cast<const char*>(v), kv_stride * es,
                     static_cast<char*>(kc), static_cast<char*>(vc), slots, row_chunks, T, num_slots);
  return hipGetLastError();
}

// ------------------------------------------------- residual + RMS Norm ----
// One wave per row, the row held in registers as fp32: r = x + residual is
// written back to `residual` (rounded once), y = r / rms(r) * w.  VPL 16-byte
// vectors per lane cover the row.
template <bool BF16, int VPL>
__global__ __launch_bounds__(256) void add_rmsnorm_kernel(const void* x, void* res, const void* __restrict__ w,
                                                          void* y, int64_t M, int H, float eps) {
  constexpr int EPV = BF16 ? 8 : 4;  // elements per 16-byte vector
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int nvec = H / EPV;
  const int64_t off = row * (int64_t)H * (BF16 ? 2 : 4);
  const u32x4* xr = reinterpret_cast<const u32x4*>(static_cast<const char*>(x) + off);
  u32x4* rr = reinterpret_cast<u32x4*>(static_cast<char*>(res) + off);
  u32x4* yr = reinterpret_cast<u32x4*>(static_cast<char*>(y) + off);
  const u32x4* wr = reinterpret_cast<const u32x4*>(w);
  auto unpack = [](const u32x4& v, float* f) {
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) f[2 * i] = bf_lo(v[i]), f[2 * i + 1] = bf_hi(v[i]);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
    }
  };
  auto pack = [](const float* f) {
    u32x4 o;
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = pack_bf2(f[2 * i], f[2 * i + 1]);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = __float_as_uint(f[i]);
    }
    return o;
  };
  float sum[VPL][EPV];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int idx = lane + i * 64;
    if (idx < nvec) {
      float a[EPV], b[EPV];
      // plain (cached) loads and stores, as in the RMS Norm kernel (faster
      // than the nontemporal forms on a streamed row block)
      unpack(xr[idx], a);
      unpack(rr[idx], b);
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        sum[i][e] = a[e] + b[e];
        ss = fmaf(sum[i][e], sum[i][e], ss);
      }
    } else {
#pragma unroll
      for (int e = 0; e < EPV; ++e) sum[i][e] = 0.f;
    }
  }
  ss = wave_sum_f(ss);
  const float r = rsqrtf(ss / (float)H + eps);
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int idx = lane + i * 64;
    if (idx >= nvec) continue;
    rr[idx] = pack(sum[i]);
    float g[EPV], o[EPV];
    unpack(wr[idx], g);
#pragma unroll
    for (int e = 0; e < EPV; ++e) o[e] = sum[i][e] * r * g[e];
    yr[idx] = pack(o);
  }
}

template <bool BF16>
static hipError_t add_rmsnorm_dispatch(const void* x, void* res, const void* w, void* y, int64_t M, int64_t H,
                                       float eps, hipStream_t s) {
  const int64_t nvec = H / (BF16 ? 8 : 4);
  const int vpl = (int)((nvec + 63) / 64);
  const dim3 grid((unsigned)((M + 3) / 4)), block(256);
  const int h = (int)H;
#define OPS_ADDRMS(V) \
  hipLaunchKernelGGL((add_rmsnorm_kernel<BF16, V>), grid, block, 0, s, x, res, w, y, M, h, eps)
  if (vpl <= 1) OPS_ADDRMS(1);
  else if (vpl <= 2) OPS_ADDRMS(2);
  else if (vpl <= 4) OPS_ADDRMS(4);
  else if (vpl <= 8) OPS_ADDRMS(8);
  else OPS_ADDRMS(16);
#undef OPS_ADDRMS
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(const void* x, void* res, const void* w, void* y, int64_t M, int64_t H, float eps,
                              bool bf16, hipStream_t s) {
  return bf16 ? add_rmsnorm_dispatch<true>(x, res, w, y, M, H, eps, s)
              : add_rmsnorm_dispatch<false>(x, res, w, y, M, H, eps, s);
}

}  // namespace opscale
