// Linear layers y[M,N] = x[M,K] W[N,K]^T (+ bias): QKV, O, gate-up and down
// projections of the decoder layer.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation.  A 256x256
// block tile is staged through LDS in BK = 64 slices with two stages; the next
// slice is fetched with buffer_load ... lds (HBM/L2 -> LDS without passing
// through registers) while the current one feeds the matrix cores.  Rows and
// K columns beyond the matrix read as zeros through the buffer descriptor's
// range check, so ragged M, N and K need no separate code path.
//
// Both operands are K-contiguous, which is what an MFMA operand lane wants: a
// lane holds 8 consecutive k of one row.  The W tile is the MFMA "A" operand
// and the x tile the "B" operand, so each accumulator lane owns one output row
// m and runs of 4 consecutive columns n, stored as 8-byte chunks.
//
// fp32 path: a plain LDS-tiled FMA kernel (exact fp32 products and sums).
#include "common.h"
#include "launch.h"

namespace opscale {

namespace {

constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kWM = 128, kWN = 64;                           // wave tile (m x n)
constexpr int kWavesM = kBM / kWM, kWavesN = kBN / kWN;      // 2 x 4
constexpr int kThreads = kWavesM * kWavesN * 64;             // 512
constexpr int kRowBytes = kBK * 2;                           // 128 B per LDS row
constexpr int kStageBytes = (kBM + kBN) * kRowBytes;         // 64 KB
constexpr int kGroupM = 8;                                   // tile rows per L2 group

// 16-byte chunk c of LDS row r lives at physical chunk c ^ swz(r).  For any 8
// consecutive rows (32-bank view) and any 16 consecutive rows (64-bank view)
// the same logical chunk lands in distinct bank groups, so the per-lane
// 16-byte fragment reads below are conflict-free.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

// Loads rows [0, rows) x k-slice [k0, k0 + 64) of a K-contiguous bf16 matrix
// (descriptor based at the tile's first row) into one LDS stage region.
// Wave w handles 8-row groups w, w + 8, ...; lane p of a group writes LDS
// bytes [p*16, p*16+16) of the group, i.e. row p/8, physical chunk p%8.
template <int ROWS>
__device__ __forceinline__ void load_tile(__amdgpu_buffer_rsrc_t rsrc, OPS_LDS char* lds, int K, int k0,
                                          int wave, int lane) {
  const int rl = lane >> 3, pc = lane & 7;
#pragma unroll
  for (int grp = wave; grp < ROWS / 8; grp += kThreads / 64) {
    const int r = grp * 8 + rl;
    const int c = pc ^ swz(r);
    const int k = k0 + c * 8;
    const uint32_t voff = k < K ? (uint32_t)(((int64_t)r * K + k) * 2) : kOobOffset;
    buffer_load16_lds(rsrc, lds + grp * 8 * kRowBytes, voff);
  }
}

__device__ __forceinline__ bf16x8 lds_frag(const OPS_LDS char* base, int r, int c) {
  return *reinterpret_cast<const OPS_LDS bf16x8*>(base + r * kRowBytes + ((c ^ swz(r)) << 4));
}

}  // namespace

__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(const __bf16* __restrict__ x,
                                                                const __bf16* __restrict__ W,
                                                                const __bf16* __restrict__ bias,
                                                                __bf16* __restrict__ y, int M, int N,
                                                                int K) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;

  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
  const uint32_t tid = xcd_remap(blockIdx.x, (uint32_t)(tiles_m * tiles_n));
  // grouped order: kGroupM tile-rows sweep the tile-columns together
  const int group = tid / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int in_group = tid % (kGroupM * tiles_n);
  const int tm = first_m + in_group % gsize, tn = in_group / gsize;
  const int m0 = tm * kBM, n0 = tn * kBN;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave % kWavesM, wn = wave / kWavesM;

  const __amdgpu_buffer_rsrc_t xr =
      make_rsrc(x + (int64_t)m0 * K, (uint32_t)(min(kBM, M - m0) * K * 2));
  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc(W + (int64_t)n0 * K, (uint32_t)(min(kBN, N - n0) * K * 2));

  f32x16 acc[kWN / 32][kWM / 32];
#pragma unroll
  for (int i = 0; i < kWN / 32; ++i)
#pragma unroll
    for (int j = 0; j < kWM / 32; ++j) acc[i][j] = f32x16{};

  const int nk = (K + kBK - 1) / kBK;
  auto stage_x = [&](int s) { return smem + s * kStageBytes; };
  auto stage_w = [&](int s) { return smem + s * kStageBytes + kBM * kRowBytes; };

  load_tile<kBM>(xr, stage_x(0), K, 0, wave, lane);
  load_tile<kBN>(wr, stage_w(0), K, 0, wave, lane);

  const int fr = lane & 31, fh = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    wait_vmem();
    __syncthreads();
    if (kt + 1 < nk) {
      load_tile<kBM>(xr, stage_x((kt + 1) & 1), K, (kt + 1) * kBK, wave, lane);
      load_tile<kBN>(wr, stage_w((kt + 1) & 1), K, (kt + 1) * kBK, wave, lane);
    }
    const OPS_LDS char* sx = stage_x(kt & 1);
    const OPS_LDS char* sw = stage_w(kt & 1);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int c = ks * 2 + fh;
      bf16x8 a[kWN / 32], b[kWM / 32];
#pragma unroll
      for (int i = 0; i < kWN / 32; ++i) a[i] = lds_frag(sw, wn * kWN + i * 32 + fr, c);
#pragma unroll
      for (int j = 0; j < kWM / 32; ++j) b[j] = lds_frag(sx, wm * kWM + j * 32 + fr, c);
#pragma unroll
      for (int i = 0; i < kWN / 32; ++i)
#pragma unroll
        for (int j = 0; j < kWM / 32; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  // Epilogue.  acc[i][j] element e: n = n0 + wn*64 + i*32 + (e/4)*8 + fh*4 + e%4,
  // m = m0 + wm*128 + j*32 + fr.  Four consecutive n per lane -> one 8-byte store.
#pragma unroll
  for (int j = 0; j < kWM / 32; ++j) {
    const int m = m0 + wm * kWM + j * 32 + fr;
    if (m >= M) continue;
    __bf16* yrow = y + (int64_t)m * N;
#pragma unroll
    for (int i = 0; i < kWN / 32; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * kWN + i * 32 + g * 8 + fh * 4;
        if (n >= N) continue;
        float v0 = acc[i][j][g * 4 + 0], v1 = acc[i][j][g * 4 + 1];
        float v2 = acc[i][j][g * 4 + 2], v3 = acc[i][j][g * 4 + 3];
        if (bias) {
          const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
          v0 += bf_lo(bb[0]);
          v1 += bf_hi(bb[0]);
          v2 += bf_lo(bb[1]);
          v3 += bf_hi(bb[1]);
        }
        u32x2 out;
        out[0] = pack_bf2(v0, v1);
        out[1] = pack_bf2(v2, v3);
        *reinterpret_cast<u32x2*>(yrow + n) = out;
      }
    }
  }
}

// ------------------------------------------------------------ fp32 path ----
// 64x64 output tile, 256 threads with 4x4 outputs each, K in slices of 16.
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ x,
                                                       const float* __restrict__ W,
                                                       const float* __restrict__ bias,
                                                       float* __restrict__ y, int M, int N, int K) {
  __shared__ float xs[16][64 + 4];
  __shared__ float ws[16][64 + 4];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + i * 256;
      const int r = idx >> 4, c = idx & 15;
      const int k = k0 + c;
      xs[c][r] = (m0 + r < M && k < K) ? x[(int64_t)(m0 + r) * K + k] : 0.f;
      ws[c][r] = (n0 + r < N && k < K) ? W[(int64_t)(n0 + r) * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = xs[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) y[(int64_t)m * N + n] = acc[i][j] + (bias ? bias[n] : 0.f);
    }
  }
}

hipError_t launch_linear(const void* x, const void* W, const void* bias, void* y, int64_t M,
                         int64_t N, int64_t K, bool bf16, hipStream_t s) {
  if (bf16) {
    // 128 KB of dynamic LDS per workgroup exceeds the default limit: raise it
    // once per process (a host-side attribute, no allocation).
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
        2 * kStageBytes);
    if (attr != hipSuccess) return attr;
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    hipLaunchKernelGGL(gemm_bf16_kernel, dim3((unsigned)tiles), dim3(kThreads), 2 * kStageBytes, s,
                       static_cast<const __bf16*>(x), static_cast<const __bf16*>(W),
                       static_cast<const __bf16*>(bias), static_cast<__bf16*>(y), (int)M, (int)N,
                       (int)K);
  } else {
    const dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
    hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, static_cast<const float*>(x),
                       static_cast<const float*>(W), static_cast<const float*>(bias),
                       static_cast<float*>(y), (int)M, (int)N, (int)K);
  }
  return hipGetLastError();
}

}  // namespace opscale
