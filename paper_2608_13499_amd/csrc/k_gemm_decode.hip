// Linear layers at decode-batch M (33 to 256 rows): y[M,N] = x[M,K] W[N,K]^T.
//
// Here every weight byte is read once from HBM and used for only M flops, so
// at M = 256 the weight stream and the matrix cores need about the same time
// (MI355X: 8 TB/s against 2.5 PFLOP/s is 312 flops per byte).  Both must stay
// busy at once, which asks for far more weight bytes in flight per CU than a
// tile ring in LDS can hold next to the activations.
//
// One workgroup of four waves (one per SIMD, up to 512 registers per lane)
// owns 128 output columns and all M rows over one K range:
//  * each wave streams its own 32 weight rows straight into registers, in
//    64-wide K slices, kAhead slices ahead of the one in use (a ring of
//    kWSlots slices, 16 VGPRs each); no LDS, no barrier on this path;
//  * the x slice of all M rows is shared through a 4-stage LDS ring filled by
//    LDS DMA (x is small and stays in L2: every workgroup reads it);
//  * MFMA 32x32x16 with the weight fragment as A (32 weight rows) and the x
//    fragment as B (32 x rows), so a lane's accumulator holds one x row and
//    four runs of four consecutive output columns (8-byte bf16 stores).
//
// Within a 64-wide slice, MFMA step j (0..3) of lane half h contracts over
// k = 32 h + 8 j + e (e < 8): each lane then loads 64 contiguous bytes of its
// weight row per slice.  The contraction index is summed over, so any
// bijection between k and the instruction's slots is valid when both operands
// use it; the x fragments are read from LDS in the same order.
//
// K is split over workgroups when the column tiles alone give fewer than
// about one workgroup per CU; the fp32 partials go to the caller's workspace
// and are summed in split order by a second kernel (deterministic).
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {

constexpr int kNumCUs = 256;
constexpr int kBK = 64;       // K per slice
constexpr int kStages = 4;    // x ring depth (LDS)
constexpr int kWSlots = 8;    // weight ring (registers)
constexpr int kAhead = 5;     // weight slices in flight beyond the one in use
constexpr int kCols = 128;    // output columns per workgroup (32 per wave)
static_assert(kAhead < kWSlots && kWSlots % kStages == 0, "ring shapes");

// 16-byte chunk c of x row r sits at chunk c ^ dswz(r) of its 128-byte LDS
// row.  An MFMA B-operand read has 32 rows (lane % 32) at one chunk per lane
// half; gfx950 serves a 16-byte read in four passes of 16 lanes (2 * (lane /
// 32) + the parity of bits 2..4 of the lane, measured), and this swizzle gives
// each pass 16 distinct 16-byte bank groups.  Depends on r mod 32 only.
__device__ __forceinline__ int dswz(int r) {
  r &= 31;
  return (r ^ (r >> 3)) & 7;
}

// One MFMA 32x32x16, then a scheduling barrier: the compiler keeps the
// order written (each MFMA followed by one fragment read of the next step),
// and still sees the MFMA, so it inserts the wait states around it.
__device__ __forceinline__ void mfma32(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

}  // namespace

// MB: 32-row blocks of x (M <= 32 * MB).  Grid: tiles_n x nsplit workgroups.
// x and W are deliberately not __restrict__: with it the compiler treats
// their loads as invariant and moves them across the fences below.
template <int MB>
__global__ __launch_bounds__(256, 1) void gemm_decode_bf16_kernel(const __bf16* x, const __bf16* W,
                                                                  const __bf16* __restrict__ bias,
                                                                  __bf16* __restrict__ y, int M, int N, int K,
                                                                  int kchunk, int tiles_n,
                                                                  float* __restrict__ part) {
  constexpr int kStageBytes = 32 * MB * 128;  // all x rows x 64 bf16
  constexpr int XL = MB;                      // 1 KB DMA loads per wave per slice (8 rows each, 4 waves)
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;

  // Consecutive ids on one XCD (so one XCD mostly reads one K range of x),
  // split-major.
  const uint32_t id = xcd_remap(blockIdx.x, gridDim.x);
  const int split = (int)(id / (uint32_t)tiles_n), tn = (int)(id % (uint32_t)tiles_n);
  const int k0 = split * kchunk;
  const int Kr = min(K - k0, kchunk);
  const int ns = Kr / kBK;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 31, h = lane >> 5;
  const int wrow0 = tn * kCols + wave * 32;  // this wave's first weight row (output column)
  const int wrows = max(0, min(32, N - wrow0));
  // rows past N and past M read as zeros (buffer range check)
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(
      W + (int64_t)min(wrow0, N - 1) * K + k0,
      wrows > 0 ? (uint32_t)(((int64_t)(wrows - 1) * K + Kr) * 2) : 0u);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x + k0, (uint32_t)(((int64_t)(M - 1) * K + Kr) * 2));
  const uint32_t w_voff = (uint32_t)((li * K + 32 * h) * 2);

  // x DMA: load g of this wave covers rows 8 (4 g + wave) .. + 7; lane p
  // writes physical chunk p % 8 of row 8 (4 g + wave) + p / 8.
  uint32_t x_voff[XL];
#pragma unroll
  for (int g = 0; g < XL; ++g) {
    const int r = (4 * g + wave) * 8 + lane / 8;
    x_voff[g] = (uint32_t)((r * K + (((lane & 7) ^ dswz(r)) << 3)) * 2);
  }
  // B-fragment read of step j: row li of each 32-row block, chunk 4 h + j.
  int frag_off[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) frag_off[j] = li * 128 + (((4 * h + j) ^ dswz(li)) << 4);

  bf16x8 wf[kWSlots][4];
  bf16x8 xf[2][MB];
  f32x16 acc[MB];
#pragma unroll
  for (int r = 0; r < MB; ++r) acc[r] = f32x16{};

  // Loads past the last slice are issued too, with an offset past the buffer
  // end (they read zeros into a stage or slot no step reads any more): every
  // step then issues the same loads, so the wait below is one constant and
  // no register of the weight ring needs a second copy.
  auto load_x = [&](int s, int stage) {
    OPS_LDS char* dst = smem + stage * kStageBytes;
#pragma unroll
    for (int g = 0; g < XL; ++g)
      buffer_load16_lds<kNoL1>(xr, dst + (4 * g + wave) * 1024,
                               s < ns ? x_voff[g] + (uint32_t)s * (kBK * 2) : kOobOffset);
  };
  auto load_w = [&](auto slot_c, int s) {
    constexpr int slot = decltype(slot_c)::value;
    const uint32_t o = s < ns ? w_voff + (uint32_t)s * (kBK * 2) : kOobOffset;
#pragma unroll
    for (int j = 0; j < 4; ++j) wf[slot][j] = __builtin_bit_cast(bf16x8, buffer_load16(wr, o + 16 * j));
  };
  auto read_one = [&](int buf, int stage, int j, int r) {
    xf[buf][r] = *reinterpret_cast<const OPS_LDS bf16x8*>(smem + stage * kStageBytes + frag_off[j] + r * 4096);
  };
  // Wait until this wave's part of x slice c + 1 has landed: the loads
  // issued after it are W(c + 2), X(c + 2), W(c + 3), X(c + 3), W(c + 4).
  // The count holds only in this issue order, which fence() fixes: the
  // compiler would otherwise move weight loads in between the DMA loads.
  auto wait_x_next = [&]() { wait_vmcnt_le<12 + 2 * XL>(); };
  auto fence = [] { asm volatile("" ::: "memory"); };

  // Prologue: the loads steps -5 .. -1 would have issued, in their order.
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  using S4 = std::integral_constant<int, 4>;
  using S5 = std::integral_constant<int, 5>;
  using S6 = std::integral_constant<int, 6>;
  using S7 = std::integral_constant<int, 7>;
  load_w(S0{}, 0);
  fence();
  load_x(0, 0);
  fence();
  load_w(S1{}, 1);
  fence();
  load_x(1, 1);
  fence();
  load_w(S2{}, 2);
  fence();
  load_x(2, 2);
  fence();
  load_w(S3{}, 3);
  fence();
  load_x(3, 3);
  fence();
  load_w(S4{}, 4);
  fence();
  wait_x_next();
  barrier_keep_loads();
#pragma unroll
  for (int r = 0; r < MB; ++r) read_one(0, 0, 0, r);

  // Step c (slot c % 8, stage c % 4): MFMA steps j = 0..3 over the 32-row
  // blocks, one fragment read of the next step after each MFMA; after j = 2,
  // wait for x slice c + 1 and barrier (every wave is done with stage c),
  // refill stage c with slice c + 4 and slot c + 5 with weight slice c + 5,
  // and read slice c + 1's first fragments under j = 3.
  auto step = [&](auto slot_c, int c) {
    constexpr int slot = decltype(slot_c)::value;
    constexpr int stage = slot % kStages;
    constexpr int nstage = (slot + 1) % kStages;
    constexpr int wslot = (slot + kAhead) % kWSlots;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int buf = j & 1;
#pragma unroll
      for (int r = 0; r < MB; ++r) {
        mfma32(acc[r], wf[slot][j], xf[buf][r]);
        read_one(buf ^ 1, stage, j + 1, r);
        sched_fence();
      }
    }
    wait_x_next();
    barrier_keep_loads();
    load_x(c + 4, stage);
    fence();
    load_w(std::integral_constant<int, wslot>{}, c + kAhead);
    fence();
#pragma unroll
    for (int r = 0; r < MB; ++r) {
      mfma32(acc[r], wf[slot][3], xf[1][r]);
      read_one(0, nstage, 0, r);
      sched_fence();
    }
  };

  // Whole rounds of kWSlots steps, every step unconditional: slices past the
  // last read as zeros (out-of-range loads), so a partial last round only
  // adds MFMAs on zeros.  Every load is then issued exactly as written (a
  // weight load that only a conditional later step used was sunk by the
  // compiler into that step, past the barriers the wait counts rely on), and
  // the accumulators have one exit from the loop.  Split K ranges are whole
  // rounds, so only a K that is not a multiple of 512 pads.
  for (int base = 0; base < ns; base += kWSlots) {
    step(S0{}, base + 0);
    step(S1{}, base + 1);
    step(S2{}, base + 2);
    step(S3{}, base + 3);
    step(S4{}, base + 4);
    step(S5{}, base + 5);
    step(S6{}, base + 6);
    step(S7{}, base + 7);
  }
  wait_vmem();

  // Epilogue through LDS (the x ring is free now): each wave writes its
  // accumulators to an fp32 tile [32 MB rows][128 columns] (16-byte chunk c of
  // row m at chunk c ^ (m mod 32): conflict-free for both sides), then every
  // thread stores 16-byte runs of whole rows, so each row of the tile leaves
  // as full cache lines.  Lane (li, h) of block r holds x row 32 r + li and
  // columns 32 wave + 8 q + 4 h + (0..3), q = 0..3.
  barrier_keep_loads();
#pragma unroll
  for (int r = 0; r < MB; ++r) {
    const int m = 32 * r + li;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = 8 * wave + 2 * q + h;
      *reinterpret_cast<OPS_LDS f32x4*>((OPS_LDS char*)smem + m * 512 + ((c ^ li) << 4)) =
          f32x4{acc[r][4 * q], acc[r][4 * q + 1], acc[r][4 * q + 2], acc[r][4 * q + 3]};
    }
  }
  __syncthreads();
  const int tc = threadIdx.x & 31;           // 16-byte chunk of a tile row: columns 4 tc .. + 3
  const int n = tn * kCols + 4 * tc;
  const bool n_ok = n < N;
  float* pbase = part ? part + (int64_t)split * M * N : nullptr;
  float b0 = 0.f, b1 = 0.f, b2 = 0.f, b3 = 0.f;
  if (!part && bias && n_ok) {
    const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
    b0 = bf_lo(bb[0]);
    b1 = bf_hi(bb[0]);
    b2 = bf_lo(bb[1]);
    b3 = bf_hi(bb[1]);
  }
#pragma unroll
  for (int i = 0; i < 4 * MB; ++i) {
    const int m = 8 * i + (threadIdx.x >> 5);
    const f32x4 v = *reinterpret_cast<const OPS_LDS f32x4*>((OPS_LDS char*)smem + m * 512 + ((tc ^ (m & 31)) << 4));
    if (m >= M || !n_ok) continue;
    if (pbase) {
      *reinterpret_cast<f32x4*>(pbase + (int64_t)m * N + n) = v;
    } else {
      *reinterpret_cast<u32x2*>(y + (int64_t)m * N + n) =
          u32x2{pack_bf2(v[0] + b0, v[1] + b1), pack_bf2(v[2] + b2, v[3] + b3)};
    }
  }
}

bool decode_linear_supported(int64_t M, int64_t N, int64_t K) {
  return M >= 1 && M <= kDecodeMaxM && K % kBK == 0 && N >= 1 && K <= (1 << 20) &&
         (int64_t)kDecodeMaxM * K * 2 < ((int64_t)1 << 31) && (int64_t)kCols * K * 2 < ((int64_t)1 << 31);
}

// Slices per K range when K is split: about one workgroup per CU, each range
// a whole number of 8-slice rounds of the weight ring.
static int64_t decode_chunk_slices(int64_t N, int64_t K) {
  const int64_t tiles = (N + kCols - 1) / kCols;
  const int64_t rounds = (K / kBK + kWSlots - 1) / kWSlots;
  const int64_t s = std::max<int64_t>(1, std::min<int64_t>(kNumCUs / tiles, rounds));
  return (rounds + s - 1) / s * kWSlots;
}

int decode_linear_splits(int64_t M, int64_t N, int64_t K) {
  (void)M;
  const int64_t c = decode_chunk_slices(N, K);
  return (int)((K / kBK + c - 1) / c);
}

size_t decode_linear_ws_bytes(int64_t M, int64_t N, int64_t K) {
  const int s = decode_linear_splits(M, N, K);
  return s > 1 ? (size_t)s * M * N * sizeof(float) : 0;
}

// splits <= 1: one K range; otherwise the ranges decode_linear_splits counts.
template <int MB>
static hipError_t launch_decode(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, int splits, float* part, hipStream_t s) {
  constexpr int lds = kStages * 32 * MB * 128;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(gemm_decode_bf16_kernel<MB>), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (N + kCols - 1) / kCols;
  const int64_t chunk = splits > 1 ? decode_chunk_slices(N, K) * kBK : K;
  const int nsplit = (int)((K + chunk - 1) / chunk);
  hipLaunchKernelGGL((gemm_decode_bf16_kernel<MB>), dim3((unsigned)(tiles * nsplit)), dim3(256), lds, s,
                     static_cast<const __bf16*>(x), static_cast<const __bf16*>(W), static_cast<const __bf16*>(bias),
                     static_cast<__bf16*>(y), (int)M, (int)N, (int)K, (int)chunk, (int)tiles,
                     nsplit > 1 ? part : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nsplit <= 1) return e;
  return launch_splitk_reduce(part, nsplit, bias, y, M, N, s);
}

hipError_t launch_linear_decode(const void* x, const void* W, const void* bias, void* y, int64_t M, int64_t N,
                                int64_t K, int splits, void* ws, hipStream_t s) {
  float* part = static_cast<float*>(ws);
  if (M <= 64) return launch_decode<2>(x, W, bias, y, M, N, K, splits, part, s);
  if (M <= 128) return launch_decode<4>(x, W, bias, y, M, N, K, splits, part, s);
  return launch_decode<8>(x, W, bias, y, M, N, K, splits, part, s);
}

}  // namespace opscale
