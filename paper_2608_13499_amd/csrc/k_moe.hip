// Mixture-of-experts FFN (the FusedMoE operator): top-k routing, and the
// routed expert SwiGLU MLPs with the routing-weighted sum.
//
// The expert MLPs run as two grouped GEMMs over the token-slot pairs sorted
// by expert, so each expert's weights are streamed once per tile-row of its
// tokens:
//   1. sort (stable, deterministic): per-block counts of each expert, one
//      exclusive scan (expert row offsets and tile offsets), then a scatter in
//      entry order, so pair i = t * topk + j lands at row pos[i] and row p of
//      the sorted list reads token gather[p];
//   2. gate_up[p] = W1[e] x[gather[p]]   (grouped GEMM, rows gathered);
//   3. act[p] = silu(gate_up[p, :F]) * gate_up[p, F:]   (the SwiGLU kernel);
//   4. y[p] = W2[e] act[p]               (grouped GEMM);
//   5. out[t] = sum_j w[t, j] y[pos[t * topk + j]], in slot order (fp32).
// Everything is ordered, so results are bitwise reproducible.
#include <algorithm>
#include <cmath>

#include <cstdlib>
#include <cstring>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr int kSortChunk = 512;  // routing entries per sort block
constexpr int kMaxExperts = 1024;

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return lane ? (~0ull >> (64 - lane)) : 0ull; }

// ---------------------------------------------------------------- routing ----
// One wave per token.  Lane l holds logits l, l + 64, ...; the softmax
// denominator uses all E logits; the k largest are taken one at a time (the
// lowest expert index among equal logits first).
template <int VPL>
__global__ __launch_bounds__(256) void moe_topk_kernel(const float* __restrict__ logits, int32_t* __restrict__ ids,
                                                       float* __restrict__ wts, int64_t T, int E, int k,
                                                       int renormalize) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* row = logits + t * E;
  float v[VPL];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int e = lane + 64 * i;
    v[i] = e < E ? row[e] : -INFINITY;
    mx = fmaxf(mx, v[i]);
  }
  mx = wave_max(mx);
  float den = 0.f;
#pragma unroll
  for (int i = 0; i < VPL; ++i)
    if (lane + 64 * i < E) den += expf(v[i] - mx);
  den = wave_sum(den);
  uint32_t taken = 0;
  float my_w = 0.f, wsum = 0.f;  // lane j keeps the j-th pick
  int my_e = 0;
  for (int j = 0; j < k; ++j) {
    // this lane's best untaken (value, index)
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int e = lane + 64 * i;
      if (e < E && !(taken >> i & 1u) && (v[i] > bv || (v[i] == bv && e < bi))) {
        bv = v[i];
        bi = e;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if ((bi & 63) == lane) taken |= 1u << (bi >> 6);
    const float w = expf(bv - mx) / den;
    if (lane == j) {
      my_w = w;
      my_e = bi;
    }
    wsum += w;
  }
  if (lane < k) {
    ids[t * k + lane] = my_e;
    wts[t * k + lane] = renormalize ? my_w / wsum : my_w;
  }
}

// ------------------------------------------------------------------- sort ----
// counts[b][e]: entries of block b routed to expert e (ids outside [0, E) are
// not counted).
__global__ __launch_bounds__(64) void moe_count_kernel(const int32_t* __restrict__ ids, int64_t R, int E,
                                                       int32_t* __restrict__ counts) {
  __shared__ int32_t cnt[kMaxExperts];
  for (int e = threadIdx.x; e < E; e += 64) cnt[e] = 0;
  __syncthreads();
  const int64_t begin = (int64_t)blockIdx.x * kSortChunk, end = min(R, begin + kSortChunk);
  for (int64_t i = begin + threadIdx.x; i < end; i += 64) {
    const int e = ids[i];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 64) counts[(int64_t)blockIdx.x * E + e] = cnt[e];
}

// counts[b][e] becomes the exclusive prefix over the blocks; rows[e] / tiles[e]
// the exclusive prefixes over the experts of the totals and of their tile
// counts (tile_rows rows per tile); rows[E], tiles[E] the sums.  16 waves:
// for 64 experts at a time, wave q sums its range of blocks, wave 0 scans, and
// each wave then writes its range's running prefixes.
__global__ __launch_bounds__(1024) void moe_scan_kernel(int32_t* __restrict__ counts, int nb, int E, int tile_rows,
                                                        int32_t* __restrict__ rows, int32_t* __restrict__ tiles) {
  constexpr int Q = 16;
  __shared__ int32_t part[Q][64];
  __shared__ int32_t carry[2];
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int per = (nb + Q - 1) / Q;
  const int b0 = q * per, b1 = min(nb, b0 + per);
  if (threadIdx.x == 0) carry[0] = carry[1] = 0;
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    int sum = 0;
    if (e < E)
      for (int b = b0; b < b1; ++b) sum += counts[(int64_t)b * E + e];
    part[q][lane] = sum;
    __syncthreads();
    if (q == 0) {
      int tot = 0;
#pragma unroll
      for (int qq = 0; qq < Q; ++qq) {
        const int c = part[qq][lane];
        part[qq][lane] = tot;  // exclusive prefix over the block ranges
        tot += c;
      }
      if (e >= E) tot = 0;
      const int nt = (tot + tile_rows - 1) / tile_rows;
      int sr = tot, st = nt;  // inclusive scans over the lanes
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int ur = __shfl_up(sr, o, 64), ut = __shfl_up(st, o, 64);
        if (lane >= o) {
          sr += ur;
          st += ut;
        }
      }
      const int cr = carry[0], ct = carry[1];
      if (e < E) {
        rows[e] = cr + sr - tot;
        tiles[e] = ct + st - nt;
      }
      const int lr = __shfl(sr, 63, 64), lt = __shfl(st, 63, 64);
      if (lane == 0) {
        carry[0] = cr + lr;
        carry[1] = ct + lt;
      }
    }
    __syncthreads();
    if (e < E) {
      int run = part[q][lane];
      for (int b = b0; b < b1; ++b) {
        const int c = counts[(int64_t)b * E + e];
        counts[(int64_t)b * E + e] = run;
        run += c;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    rows[E] = carry[0];
    tiles[E] = carry[1];
  }
}

// Entries of block b in order: entry i (token i / topk) routed to expert e
// goes to sorted row rows[e] + counts[b][e] + (its rank among block b's
// earlier entries of expert e).  pos[i] = -1 for ids outside [0, E).
__global__ __launch_bounds__(64) void moe_scatter_kernel(const int32_t* __restrict__ ids, int64_t R, int E, int k,
                                                         const int32_t* __restrict__ counts,
                                                         const int32_t* __restrict__ rows,
                                                         int32_t* __restrict__ gather, int32_t* __restrict__ pos) {
  __shared__ int32_t next[kMaxExperts];
  const int lane = threadIdx.x;
  for (int e = lane; e < E; e += 64) next[e] = rows[e] + counts[(int64_t)blockIdx.x * E + e];
  __syncthreads();
  const int64_t begin = (int64_t)blockIdx.x * kSortChunk, end = min(R, begin + kSortChunk);
  for (int64_t base = begin; base < end; base += 64) {
    const int64_t i = base + lane;
    const bool valid = i < end;
    const int e = valid ? ids[i] : -1;
    const bool ok = valid && e >= 0 && e < E;
    if (valid && !ok) pos[i] = -1;
    uint64_t todo = __builtin_amdgcn_ballot_w64(ok);
    while (todo) {
      const int leader = __builtin_amdgcn_readfirstlane(__builtin_ctzll(todo));
      const int el = __builtin_amdgcn_readlane(e, leader);
      const bool mine = ok && e == el;
      const uint64_t m = __builtin_amdgcn_ballot_w64(mine);
      const int start = next[el];
      if (mine) {
        const int p = start + __builtin_popcountll(m & lanemask_lt(lane));
        gather[p] = (int32_t)(i / k);
        pos[i] = p;
      }
      __syncthreads();  // every lane has read next[el] (one wave: a wait, not a barrier)
      if (lane == leader) next[el] = start + __builtin_popcountll(m);
      __syncthreads();
      todo &= ~m;
    }
  }
}

// ---------------------------------------------------------------- combine ----
// out[t] = sum_j w[t, j] y[pos[t * k + j]] (slots in order, fp32), 8 columns per
// thread.
__global__ __launch_bounds__(256) void moe_combine_kernel(const __bf16* __restrict__ y, const int32_t* __restrict__ pos,
                                                          const float* __restrict__ wts, __bf16* __restrict__ out,
                                                          int H, int k) {
  const int64_t t = blockIdx.x;
  for (int c = threadIdx.x * 8; c < H; c += 256 * 8) {
    float acc[8] = {};
    for (int j = 0; j < k; ++j) {
      const int p = pos[t * k + j];
      if (p < 0) continue;
      const float w = wts[t * k + j];
      const u32x4 v = *reinterpret_cast<const u32x4*>(y + (int64_t)p * H + c);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += w * bf_lo(v[q]);
        acc[2 * q + 1] += w * bf_hi(v[q]);
      }
    }
    *reinterpret_cast<u32x4*>(out + t * H + c) =
        u32x4{pack_bf2(acc[0], acc[1]), pack_bf2(acc[2], acc[3]), pack_bf2(acc[4], acc[5]), pack_bf2(acc[6], acc[7])};
  }
}

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct MoeWorkspace {
  int32_t *counts, *rows, *tiles, *gather, *pos;
  __bf16 *gate_up, *act, *y;
  size_t bytes;
};

MoeWorkspace carve(void* base, int64_t T, int H, int F, int E, int k) {
  const int64_t R = T * k;
  const int64_t nb = (R + kSortChunk - 1) / kSortChunk;
  MoeWorkspace w{};
  char* p = static_cast<char*>(base);
  size_t off = 0;
  auto take = [&](size_t b) {
    char* q = p ? p + off : nullptr;
    off += align256(b);
    return q;
  };
  w.counts = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)std::max<int64_t>(1, nb) * E));
  w.rows = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)(E + 1)));
  w.tiles = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)(E + 1)));
  w.gather = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)R));
  w.pos = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)R));
  w.gate_up = reinterpret_cast<__bf16*>(take(2 * (size_t)R * 2 * F));
  w.act = reinterpret_cast<__bf16*>(take(2 * (size_t)R * F));
  w.y = reinterpret_cast<__bf16*>(take(2 * (size_t)R * H));
  w.bytes = off;
  return w;
}
}  // namespace

int32_t moe_max_experts() { return kMaxExperts; }

size_t moe_workspace_bytes(int64_t T, int32_t H, int32_t F, int32_t E, int32_t topk) {
  return carve(nullptr, T, H, F, E, topk).bytes;
}

hipError_t launch_moe_topk(const float* logits, int32_t* ids, float* wts, int64_t T, int32_t E, int32_t k,
                           bool renormalize, hipStream_t s) {
  const dim3 grid((unsigned)((T + 3) / 4)), block(256);
  const int vpl = (E + 63) / 64;
#define OPS_TOPK(V) \
  hipLaunchKernelGGL((moe_topk_kernel<V>), grid, block, 0, s, logits, ids, wts, T, E, k, (int)renormalize)
  if (vpl <= 1) OPS_TOPK(1);
  else if (vpl <= 2) OPS_TOPK(2);
  else if (vpl <= 4) OPS_TOPK(4);
  else if (vpl <= 8) OPS_TOPK(8);
  else OPS_TOPK(16);
#undef OPS_TOPK
  return hipGetLastError();
}

hipError_t launch_fused_moe(const void* x, const void* w1, const void* w2, const int32_t* ids, const float* wts,
                            void* out, int64_t T, int32_t H, int32_t F, int32_t E, int32_t k, void* ws,
                            hipStream_t s) {
  const int64_t R = T * k;
  const int nb = (int)((R + kSortChunk - 1) / kSortChunk);
  const MoeWorkspace w = carve(ws, T, H, F, E, k);
  const int32_t bm = grouped_gemm_tile_rows(R, E);
  hipLaunchKernelGGL(moe_count_kernel, dim3((unsigned)nb), dim3(64), 0, s, ids, R, E, w.counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(moe_scan_kernel, dim3(1), dim3(1024), 0, s, w.counts, nb, E, bm, w.rows, w.tiles);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(moe_scatter_kernel, dim3((unsigned)nb), dim3(64), 0, s, ids, R, E, k, w.counts, w.rows, w.gather,
                     w.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // act = silu(W1g[e] x[token]) * (W1u[e] x[token])   (rows gathered), [R, F]:
  // the SwiGLU sits in the GEMM's epilogue when an expert's gate-up weight
  // spans less than 4 GB (32-bit row offsets); else gate_up [R, 2F] first
  // (OPSCALE_TUNE_MOE_FUSE = 0 forces the unfused path, for tests)
  if ((int64_t)2 * F * H * 2 < ((int64_t)1 << 32) && tuning(OPSCALE_TUNE_MOE_FUSE) != 0) {
    if ((e = launch_gemm_grouped(x, T, w1, (int64_t)2 * F * H, w.act, R, 2 * (int64_t)F, H, E, bm, w.gather, w.rows,
                                 w.tiles, F, s)) != hipSuccess)
      return e;
  } else {
    if ((e = launch_gemm_grouped(x, T, w1, (int64_t)2 * F * H, w.gate_up, R, 2 * (int64_t)F, H, E, bm, w.gather,
                                 w.rows, w.tiles, 0, s)) != hipSuccess)
      return e;
    if ((e = launch_swiglu(w.gate_up, w.act, R, F, true, s)) != hipSuccess) return e;
  }
  // y = W2[e] act   (sorted rows), [R, H]
  if ((e = launch_gemm_grouped(w.act, R, w2, (int64_t)H * F, w.y, R, H, F, E, bm, nullptr, w.rows, w.tiles, 0, s)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(moe_combine_kernel, dim3((unsigned)T), dim3(256), 0, s, w.y, w.pos, wts,
                     static_cast<__bf16*>(out), H, k);
  return hipGetLastError();
}

}  // namespace opscale
