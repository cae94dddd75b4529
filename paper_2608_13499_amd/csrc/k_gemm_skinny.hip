// Linear layers at small M: y[M,N] = x[M,K] W[N,K]^T (+ bias) when M is a
// decode batch (one row per sequence).  Then the weights dominate the traffic
// (M flops per weight byte) and the tiled GEMM's 256x256 tiles would give only
// N / 256 workgroups.  Here one workgroup of 8 waves owns 16 x NG output
// columns and all M rows; its waves split K, each streaming a contiguous K
// range of the workgroup's weight rows with MFMA 16x16x32 (x as the A operand,
// 16 rows per group, MG groups; W as the B operand), and the 8 partial tiles
// are summed through LDS in a fixed order, so results are deterministic.
// Requires K % 32 == 0 and M <= 16 * MG.
#include <cstdlib>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr int kSkinnyWaves = 8;
}  // namespace

template <int MG, int NG, int P>
__global__ __launch_bounds__(512) void gemm_skinny_bf16_kernel(const __bf16* __restrict__ x,
                                                               const __bf16* __restrict__ W,
                                                               const __bf16* __restrict__ bias,
                                                               __bf16* __restrict__ y, int M, int N, int K,
                                                               int ksteps_per_wave) {
  constexpr int NT = 16 * NG;   // output columns of the workgroup
  constexpr int T = MG * NG;    // 16x16 output tiles
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int n0 = blockIdx.x * NT;
  const int nrows = min(NT, N - n0);
  // weight rows past N and activation rows past M read as zeros
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(W + (int64_t)n0 * K, (uint32_t)((int64_t)nrows * K * 2));
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)((int64_t)M * K * 2));
  // fragment lane roles (16x16x32): row lane % 16, K elements 8 (lane / 16) .. + 8
  const int fr = lane & 15, kq = lane >> 4;
  const int ks0 = wave * ksteps_per_wave;
  const int ks1 = min(K / 32, ks0 + ksteps_per_wave);

  uint32_t xo[MG], wo[NG];
#pragma unroll
  for (int g = 0; g < MG; ++g) xo[g] = (uint32_t)(((g * 16 + fr) * K + kq * 8) * 2);
#pragma unroll
  for (int h = 0; h < NG; ++h) wo[h] = (uint32_t)(((h * 16 + fr) * K + kq * 8) * 2);

  f32x4 acc[MG][NG];
#pragma unroll
  for (int g = 0; g < MG; ++g)
#pragma unroll
    for (int h = 0; h < NG; ++h) acc[g][h] = f32x4{};

  // a ring of P k-steps of fragments in flight
  bf16x8 xf[P][MG], wf[P][NG];
  auto load = [&](int slot, int ks) {
    const uint32_t kb = (uint32_t)ks * 64u;  // 32 bf16 per k-step
#pragma unroll
    for (int h = 0; h < NG; ++h) wf[slot][h] = __builtin_bit_cast(bf16x8, buffer_load16(wr, wo[h] + kb));
#pragma unroll
    for (int g = 0; g < MG; ++g) xf[slot][g] = __builtin_bit_cast(bf16x8, buffer_load16(xr, xo[g] + kb));
  };
#pragma unroll
  for (int s = 0; s < P; ++s)
    if (ks0 + s < ks1) load(s, ks0 + s);
  for (int ks = ks0; ks < ks1; ks += P) {
#pragma unroll
    for (int s = 0; s < P; ++s) {
      if (ks + s < ks1) {
#pragma unroll
        for (int g = 0; g < MG; ++g)
#pragma unroll
          for (int h = 0; h < NG; ++h)
            acc[g][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf[s][g], wf[s][h], acc[g][h], 0, 0, 0);
        if (ks + s + P < ks1) load(s, ks + s + P);
      }
    }
  }

  // Sum the 8 waves' partial tiles, four tiles per round.  A tile's lane l
  // holds rows 4 (l / 16) + v (v < 4) of column l % 16.
  __shared__ __attribute__((aligned(16))) float red[kSkinnyWaves][4][64][4];
#pragma unroll
  for (int t0 = 0; t0 < T; t0 += 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (t0 + j < T) *reinterpret_cast<f32x4*>(&red[wave][j][lane][0]) = acc[(t0 + j) / NG][(t0 + j) % NG];
    __syncthreads();
    for (int o = threadIdx.x; o < 4 * 256; o += 512) {
      const int j = o >> 8, e = o & 255;
      const int t = t0 + j;
      if (t >= T) continue;
      const int i = e >> 4, c = e & 15;          // row and column within the tile
      const int ln = 16 * (i >> 2) + c, v = i & 3;
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < kSkinnyWaves; ++w) sum += red[w][j][ln][v];
      const int m = (t / NG) * 16 + i, n = n0 + (t % NG) * 16 + c;
      if (m < M && n < N) {
        if (bias) sum += (float)bias[n];
        y[(int64_t)m * N + n] = (__bf16)sum;
      }
    }
    __syncthreads();
  }
}

template <int MG, int NG, int P>
static hipError_t launch_skinny(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, hipStream_t s) {
  constexpr int NT = 16 * NG;
  const int ksteps = (int)(K / 32);
  const int per_wave = (ksteps + kSkinnyWaves - 1) / kSkinnyWaves;
  hipLaunchKernelGGL((gemm_skinny_bf16_kernel<MG, NG, P>), dim3((unsigned)((N + NT - 1) / NT)),
                     dim3(64 * kSkinnyWaves), 0, s, static_cast<const __bf16*>(x), static_cast<const __bf16*>(W),
                     static_cast<const __bf16*>(bias), static_cast<__bf16*>(y), (int)M, (int)N, (int)K, per_wave);
  return hipGetLastError();
}

bool skinny_linear_supported(int64_t M, int64_t N, int64_t K) {
  return M >= 1 && M <= kSkinnyMaxM && K % 32 == 0 && N >= 1;
}

// Measured on MI355X over the 8B-layer shapes at M = 1 ... 512 (cold caches):
// this path wins at M <= 16 for every shape, and at M <= 32 wherever the
// tiled GEMM has few 256x256 tiles (QKV, O, down: 16-24); beyond that the
// split-K tiled GEMM wins (and with many tiles, gate-up's 112, the plain one).
bool skinny_linear_preferred(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + 255) / 256) * ((N + 255) / 256);
  return skinny_linear_supported(M, N, K) && (M <= 16 || (M <= 32 && tiles < 64));
}

hipError_t launch_linear_skinny(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, hipStream_t s) {
  // Every workgroup reads all of x, so x is read ceil(N / 16 NG) times, M / 16 NG
  // times the weight bytes.  32 columns per workgroup (NG = 2) halve that and
  // win from M = 16 on while they still give >= 192 workgroups; otherwise the
  // extra workgroups of NG = 1 win.  OPSCALE_TUNE_SKINNY_NG forces it.
  const int32_t forced = tuning(OPSCALE_TUNE_SKINNY_NG);
  const int ng = forced == 1 || forced == 2 ? forced : (M >= 16 && (N + 31) / 32 >= 192 ? 2 : 1);
  if (ng == 2) {
    if (M <= 16) return launch_skinny<1, 2, 4>(x, W, bias, y, M, N, K, s);
    if (M <= 32) return launch_skinny<2, 2, 4>(x, W, bias, y, M, N, K, s);
    if (M <= 64) return launch_skinny<4, 2, 2>(x, W, bias, y, M, N, K, s);
    if (M <= 128) return launch_skinny<8, 2, 2>(x, W, bias, y, M, N, K, s);
    return launch_skinny<16, 2, 1>(x, W, bias, y, M, N, K, s);
  }
  if (M <= 16) return launch_skinny<1, 1, 8>(x, W, bias, y, M, N, K, s);
  if (M <= 32) return launch_skinny<2, 1, 4>(x, W, bias, y, M, N, K, s);
  if (M <= 64) return launch_skinny<4, 1, 4>(x, W, bias, y, M, N, K, s);
  if (M <= 128) return launch_skinny<8, 1, 2>(x, W, bias, y, M, N, K, s);
  return launch_skinny<16, 1, 2>(x, W, bias, y, M, N, K, s);
}

}  // namespace opscale
