// Decode attention: one new query token per sequence against its paged KV
// cache [num_blocks, block_size, Hkv, D].
//
// bf16 path.  The key range of every sequence is cut into splits of about
// kChunk keys (split-KV), so that 256 sequences x 8 KV heads give thousands of
// independent workgroups and the long and short contexts balance.  A
// workgroup (4 waves) owns one (split, KV head, sequence) and serves all G
// query heads of that KV head, so each cached K/V row is read from HBM once.
// A wave takes 32 keys at a time:
//   * scores: S^T[key][head] = K Q^T on MFMA 16x16x32 (A = 16 cached K rows
//     loaded straight from HBM into operand registers, B = the G query rows,
//     zero-padded to 16 columns);
//   * online softmax per head in the log2 domain;
//   * values: lanes own 8 consecutive head-dim columns of one key row (16-byte
//     coalesced loads) and accumulate p * v in fp32 for the G heads, the
//     probabilities broadcast through LDS.
// Each split leaves (max, sum, unnormalized output) in the caller workspace;
// a second kernel merges the splits of a (sequence, head) in split order, so
// the result is deterministic.
//
// fp32 path: one wave per (sequence, head), exact expf, no workspace use.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kChunk = 512;  // nominal keys per split, and keys per page window
constexpr int kTile = 32;    // keys per wave step
// Page ids of one window of kChunk keys (any block size >= 1) fit in here.
constexpr int kMaxPages = kChunk + 1;

struct SplitPlan {
  int n, splits, chunk;
};

// Splits of one sequence: at most max_splits, each a multiple of kTile keys.
__device__ __forceinline__ SplitPlan plan_splits(int n, int max_splits) {
  SplitPlan p;
  p.n = n;
  p.splits = n <= 0 ? 0 : min(max_splits, (n + kChunk - 1) / kChunk);
  const int per = p.splits > 0 ? (n + p.splits - 1) / p.splits : 0;
  p.chunk = (per + kTile - 1) / kTile * kTile;
  return p;
}
}  // namespace

int32_t decode_max_splits(int32_t max_context_len) {
  return std::max<int32_t>(1, (max_context_len + kChunk - 1) / kChunk);
}

size_t decode_workspace_bytes(int32_t B, int32_t Hq, int32_t D, int32_t max_context_len) {
  return (size_t)4 * (size_t)B * (size_t)Hq * (size_t)decode_max_splits(max_context_len) *
         (size_t)(D + 2);
}

template <int D, int G>
__global__ __launch_bounds__(256) void attn_decode_split_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ kc, const __bf16* __restrict__ vc,
    const int32_t* __restrict__ table, const int32_t* __restrict__ ctx, int Hq, int Hkv,
    int log2bs, int max_blocks, int64_t num_blocks, int max_splits, float scale_log2,
    float* __restrict__ ws_o, float* __restrict__ ws_ml) {
  constexpr int CPR = D / 8;        // 16-byte chunks per cache row
  constexpr int RPI = 64 / CPR;     // rows per wave load instruction (V layout)
  constexpr int KSTEPS = D / 32;    // MFMA k-steps over the head dim
  constexpr int NV = kTile / RPI;   // V loads per lane per tile
  __shared__ int32_t pages[kMaxPages];  // physical blocks of the current key window
  __shared__ float p_lds[4][G][kTile];
  __shared__ float red_m[4][G], red_l[4][G];
  __shared__ float red_o[4][G][D];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int bs = 1 << log2bs;
  const int n = min(ctx[b], max_blocks << log2bs);
  const SplitPlan plan = plan_splits(n, max_splits);
  const int k_begin = split * plan.chunk;
  if (split >= plan.splits || k_begin >= n) return;
  const int k_end = min(n, k_begin + plan.chunk);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int64_t row_elems = (int64_t)Hkv * D;

  // Page ids are looked up once per window of kChunk keys (normally the whole
  // split) and kept in LDS, so the per-tile K/V loads do not wait on a
  // dependent block-table load.  Invalid ids become -1 (rows of zeros).
  const int32_t* trow = table + (int64_t)b * max_blocks;
  int p_first = 0, w_end = 0;
  auto load_pages = [&](int w0) {
    w_end = min(k_end, w0 + kChunk);
    p_first = w0 >> log2bs;
    const int p_count = ((w_end - 1) >> log2bs) - p_first + 1;
    for (int i = threadIdx.x; i < p_count; i += 256) {
      const int blk = trow[p_first + i];
      pages[i] = (uint32_t)blk < (uint64_t)num_blocks ? blk : -1;
    }
  };

  // Query heads of this group as the MFMA B operand (column = head).
  bf16x8 qf[KSTEPS];
  {
    const bool has = col < G;
    const __bf16* qrow = q + ((int64_t)b * Hq + (int64_t)g * G + (has ? col : 0)) * D;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (has) w = *reinterpret_cast<const u32x4*>(qrow + s * 32 + grp * 8);
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // address of cache row j (absolute key index) for this KV head, or null
  auto row_ptr = [&](const __bf16* cache, int j) -> const __bf16* {
    if (j >= w_end) return nullptr;
    const int blk = pages[(j >> log2bs) - p_first];
    if (blk < 0) return nullptr;
    return cache + ((int64_t)blk * bs + (j & (bs - 1))) * row_elems + (int64_t)g * D;
  };

  // K in MFMA A-operand layout (lane: key col, 8 head-dim values at 32*s + 8*grp)
  // and V in row layout (lane: key vrow + RPI*i, 8 head-dim values at 8*vchunk).
  const int vrow = lane / CPR, vchunk = lane % CPR;
  struct TileRegs {
    u32x4 k[2][KSTEPS];
    u32x4 v[NV];
  };
  auto load_tile = [&](int t0, TileRegs& r) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const __bf16* kr = row_ptr(kc, t0 + sub * 16 + col);
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        r.k[sub][s] = kr ? *reinterpret_cast<const u32x4*>(kr + s * 32 + grp * 8) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const __bf16* vr = row_ptr(vc, t0 + i * RPI + vrow);
      r.v[i] = vr ? *reinterpret_cast<const u32x4*>(vr + vchunk * 8) : u32x4{0u, 0u, 0u, 0u};
    }
  };

  float m_run = -INFINITY, l_run = 0.f;  // for head `col` (lanes col < G meaningful)
  float acc[G][8];
#pragma unroll
  for (int hh = 0; hh < G; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[hh][e] = 0.f;

  auto compute_tile = [&](int t0, const TileRegs& r) {
    // scores S^T[key][head]: lane holds head `col`, keys t0 + 16*sub + 4*grp + rr
    f32x4 st[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      st[sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        st[sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, r.k[sub][s]), qf[s],
                                                          st[sub], 0, 0, 0);
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int j = t0 + sub * 16 + grp * 4 + rr;
        const float sv = j < w_end ? st[sub][rr] * scale_log2 : -INFINITY;
        st[sub][rr] = sv;
        tmax = fmaxf(tmax, sv);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float p = fast_exp2(st[sub][rr] - m_use);
        psum += p;
        if (col < G) p_lds[wave][col][sub * 16 + grp * 4 + rr] = p;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
      const float a = __shfl(alpha, hh, 64);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[hh][e] *= a;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // values: acc[hh][e] += p[hh][key] * v[key][vchunk*8 + e]
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int kl = i * RPI + vrow;
      float vf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[2 * e] = bf_lo(r.v[i][e]);
        vf[2 * e + 1] = bf_hi(r.v[i][e]);
      }
#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        const float p = p_lds[wave][hh][kl];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[hh][e] = fmaf(p, vf[e], acc[hh][e]);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // Software pipeline: the loads of the wave's next tile are in flight while
  // the current one is scored and accumulated.
  TileRegs cur, nxt;
  for (int w0 = k_begin; w0 < k_end; w0 += kChunk) {
    if (w0 != k_begin) __syncthreads();  // every wave is done with the previous window
    load_pages(w0);
    __syncthreads();
    int t0 = w0 + wave * kTile;
    if (t0 < w_end) load_tile(t0, cur);
    while (t0 < w_end) {
      const int t1 = t0 + 4 * kTile;
      if (t1 < w_end) load_tile(t1, nxt);
      compute_tile(t0, cur);
      cur = nxt;
      t0 = t1;
    }
  }

  // ---- merge the lanes that hold different keys of the same columns
#pragma unroll
  for (int hh = 0; hh < G; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float a = acc[hh][e];
#pragma unroll
      for (int off = CPR; off < 64; off <<= 1) a += __shfl_xor(a, off, 64);
      acc[hh][e] = a;
    }
  if (lane < CPR) {
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
      for (int e = 0; e < 8; ++e) red_o[wave][hh][lane * 8 + e] = acc[hh][e];
  }
  if (lane < G) {
    red_m[wave][lane] = m_run;
    red_l[wave][lane] = l_run;
  }
  __syncthreads();
  // ---- merge the 4 waves and write this split's partial result
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int hh = idx / D, d = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, red_m[w][hh]);
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = red_m[w][hh] == -INFINITY ? 0.f : fast_exp2(red_m[w][hh] - M);
      o += f * red_o[w][hh][d];
      l += f * red_l[w][hh];
    }
    const int h = g * G + hh;
    const int64_t slot = ((int64_t)b * Hq + h) * max_splits + split;
    ws_o[slot * D + d] = o;
    if (d == 0) {
      ws_ml[slot * 2 + 0] = M;
      ws_ml[slot * 2 + 1] = l;
    }
  }
}

// Merge the splits of one (sequence, head); one wave per pair.
template <int D>
__global__ __launch_bounds__(64) void attn_decode_combine_kernel(
    const float* __restrict__ ws_o, const float* __restrict__ ws_ml, const int32_t* __restrict__ ctx,
    __bf16* __restrict__ o, int Hq, int log2bs, int max_blocks, int max_splits) {
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int n = min(ctx[b], max_blocks << log2bs);
  const SplitPlan plan = plan_splits(n, max_splits);
  const int64_t slot0 = ((int64_t)b * Hq + h) * max_splits;
  float M = -INFINITY;
  for (int s = 0; s < plan.splits; ++s)
    if (s * plan.chunk < n) M = fmaxf(M, ws_ml[(slot0 + s) * 2]);
  float acc[D / 64] = {};
  float l = 0.f;
  for (int s = 0; s < plan.splits; ++s) {
    if (s * plan.chunk >= n) continue;
    const float f = fast_exp2(ws_ml[(slot0 + s) * 2] - M);
    l += f * ws_ml[(slot0 + s) * 2 + 1];
#pragma unroll
    for (int c = 0; c < D / 64; ++c) acc[c] += f * ws_o[(slot0 + s) * D + lane + c * 64];
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int c = 0; c < D / 64; ++c) o[((int64_t)b * Hq + h) * D + lane + c * 64] = (__bf16)(acc[c] * inv);
}

// ------------------------------------------------------------ fp32 path ----
template <int D>
__global__ __launch_bounds__(64) void attn_decode_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc, const float* __restrict__ vc,
    const int32_t* __restrict__ table, const int32_t* __restrict__ ctx, float* __restrict__ o,
    int Hq, int Hkv, int log2bs, int max_blocks, int64_t num_blocks, float scale) {
  constexpr int DPL = D / 64;
  __shared__ float qs[D];
  __shared__ float ps[64];
  __shared__ int64_t rows[64];
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int g = h / (Hq / Hkv);
  const int bs = 1 << log2bs;
  const int n = min(ctx[b], max_blocks << log2bs);
  const int32_t* trow = table + (int64_t)b * max_blocks;
  for (int d = lane; d < D; d += 64) qs[d] = q[((int64_t)b * Hq + h) * D + d];
  __syncthreads();
  float m_run = -INFINITY, l_run = 0.f, acc[DPL] = {};
  for (int kv0 = 0; kv0 < n; kv0 += 64) {
    const int j = kv0 + lane;
    float s = -INFINITY;
    int64_t row = -1;
    if (j < n) {
      const int blk = trow[j >> log2bs];
      if ((uint32_t)blk < (uint64_t)num_blocks)
        row = (((int64_t)blk * bs + (j & (bs - 1))) * Hkv + g) * D;
      float dot = 0.f;
      if (row >= 0)
        for (int d = 0; d < D; ++d) dot = fmaf(qs[d], kc[row + d], dot);
      s = dot * scale;
    }
    rows[lane] = row;
    const float m_new = fmaxf(m_run, wave_max(s));
    const float p = j < n ? expf(s - m_new) : 0.f;
    const float alpha = expf(m_run - m_new);
    l_run = l_run * alpha + wave_sum(p);
    m_run = m_new;
    ps[lane] = p;
    __syncthreads();
    const int cnt = min(64, n - kv0);
#pragma unroll
    for (int c = 0; c < DPL; ++c) {
      float a = acc[c] * alpha;
      for (int jj = 0; jj < cnt; ++jj)
        if (rows[jj] >= 0) a = fmaf(ps[jj], vc[rows[jj] + lane + c * 64], a);
      acc[c] = a;
    }
    __syncthreads();
  }
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
  for (int c = 0; c < DPL; ++c) o[((int64_t)b * Hq + h) * D + lane + c * 64] = acc[c] * inv;
}

hipError_t launch_attn_decode(const void* q, const void* kcache, const void* vcache,
                              const int32_t* table, const int32_t* ctx, void* o, int32_t B,
                              int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size,
                              int32_t max_blocks, int64_t num_blocks, int32_t max_context_len,
                              float scale, bool bf16, void* ws, hipStream_t s) {
  int log2bs = 0;
  while ((1 << log2bs) < block_size) ++log2bs;
  if (!bf16) {
    const dim3 grid((unsigned)Hq, (unsigned)B);
    if (D == 128)
      hipLaunchKernelGGL((attn_decode_f32_kernel<128>), grid, dim3(64), 0, s,
                         static_cast<const float*>(q), static_cast<const float*>(kcache),
                         static_cast<const float*>(vcache), table, ctx, static_cast<float*>(o), Hq,
                         Hkv, log2bs, max_blocks, num_blocks, scale);
    else
      hipLaunchKernelGGL((attn_decode_f32_kernel<64>), grid, dim3(64), 0, s,
                         static_cast<const float*>(q), static_cast<const float*>(kcache),
                         static_cast<const float*>(vcache), table, ctx, static_cast<float*>(o), Hq,
                         Hkv, log2bs, max_blocks, num_blocks, scale);
    return hipGetLastError();
  }
  const int max_splits = decode_max_splits(max_context_len);
  float* ws_o = static_cast<float*>(ws);
  float* ws_ml = ws_o + (size_t)B * Hq * max_splits * D;
  const dim3 grid((unsigned)max_splits, (unsigned)Hkv, (unsigned)B);
  const float sl2 = scale * kLog2e;
  const int G = Hq / Hkv;
#define OPS_DEC(DD, GG)                                                                          \
  hipLaunchKernelGGL((attn_decode_split_kernel<DD, GG>), grid, dim3(256), 0, s,                  \
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(kcache),          \
                     static_cast<const __bf16*>(vcache), table, ctx, Hq, Hkv, log2bs, max_blocks, \
                     num_blocks, max_splits, sl2, ws_o, ws_ml)
#define OPS_DEC_G(DD)                 \
  switch (G) {                        \
    case 1: OPS_DEC(DD, 1); break;    \
    case 2: OPS_DEC(DD, 2); break;    \
    case 4: OPS_DEC(DD, 4); break;    \
    default: OPS_DEC(DD, 8); break;   \
  }
  if (D == 128) {
    OPS_DEC_G(128)
  } else {
    OPS_DEC_G(64)
  }
#undef OPS_DEC_G
#undef OPS_DEC
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cgrid((unsigned)Hq, (unsigned)B);
  if (D == 128)
    hipLaunchKernelGGL((attn_decode_combine_kernel<128>), cgrid, dim3(64), 0, s, ws_o, ws_ml, ctx,
                       static_cast<__bf16*>(o), Hq, log2bs, max_blocks, max_splits);
  else
    hipLaunchKernelGGL((attn_decode_combine_kernel<64>), cgrid, dim3(64), 0, s, ws_o, ws_ml, ctx,
                       static_cast<__bf16*>(o), Hq, log2bs, max_blocks, max_splits);
  return hipGetLastError();
}

}  // namespace opscale
