// Decode attention: one new query token per sequence against its paged KV
// cache [num_blocks, block_size, Hkv, D].
//
// bf16 path.  The key range of every sequence is cut into splits (split-KV) of
// 32 ... 512 keys, the size chosen per launch so that the batch gives about
// 1024 workgroups: 256 sequences of thousands of keys get 512-key splits,
// a single sequence 32-key ones, and long and short contexts balance.  A workgroup of 8 waves owns one (split,
// sequence, group of up to 8 KV heads): for the 8-head layer every wave takes
// one KV head and serves all G query heads of that head, so each page of the
// cache (block_size slots x all heads, contiguous) is streamed by one
// workgroup in one pass and each K/V row is read from HBM exactly once.
// Per 32 keys a wave does:
//   * scores S^T[key][head] = K Q^T on MFMA 16x16x32: A = 16 cached K rows
//     loaded straight from HBM into operand registers, B = the G query rows
//     zero-padded to 16 columns;
//   * online softmax per head in the log2 domain (lazy reference max);
//   * O[head][d] += P V on MFMA 16x16x32: the S^T accumulator is already the
//     A operand P (a lane holds one head and 8 keys), and V, DMA'd into LDS
//     row-major, is read as the B operand with ds_read_b64_tr_b16.
// A wave loads a tile and waits for it; the latency is covered by the other
// waves of the CU: with one V buffer per wave (64 KB of LDS) and at most 128
// VGPRs, two workgroups (16 waves) share a CU.  V is read with the
// nontemporal hint, the cache is streamed once.
// Each split leaves (max, sum, unnormalized output) in the caller workspace; a
// second kernel merges the splits of a (sequence, head) in split order, so the
// result is deterministic.
//
// Keys whose page id is outside [0, num_blocks) are skipped.
//
// fp32 path: one wave per (sequence, head), exact expf, no workspace use.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kChunk = 512;  // the largest split, and keys per page window
constexpr int kFillWorkgroups = 1024;  // splits are sized to give about this many
constexpr int kMaxSplitsForFill = 64;   // ... but a sequence gets at most this many
constexpr int kTile = 32;    // keys per wave step
constexpr int kWaves = 8;    // waves per workgroup
// Page ids of one window of kChunk keys (any block size >= 1) fit in here.
constexpr int kMaxPages = kChunk + 1;

struct SplitPlan {
  int n, splits, chunk;
};

// Splits of one sequence: about chunk_keys keys each, at most max_splits,
// each a multiple of kTile keys.
__device__ __forceinline__ SplitPlan plan_splits(int n, int max_splits, int chunk_keys) {
  SplitPlan p;
  p.n = n;
  p.splits = n <= 0 ? 0 : min(max_splits, (n + chunk_keys - 1) / chunk_keys);
  const int per = p.splits > 0 ? (n + p.splits - 1) / p.splits : 0;
  p.chunk = (per + kTile - 1) / kTile * kTile;
  return p;
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// gfx950 transposed LDS read: within each 16-lane group, lane i receives
// element i % 4 of the 8-byte chunks addressed by lanes 4e + i / 4 (e = 0..3).
__device__ __forceinline__ u32x2 lds_read_tr16(const OPS_LDS char* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((OPS_LDS s16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// V rows in LDS: the 16-byte chunk c of row r sits at chunk c ^ v_swz(r), so
// the 4 rows x 32 bytes a 16-lane group reads with one transposed read fall
// into distinct bank groups.
__device__ __forceinline__ int v_swz(int r) { return (r & 3) << 1; }
}  // namespace

int32_t decode_chunk_keys(int32_t B, int32_t max_context_len) {
  const int64_t ctx = std::max(1, max_context_len);
  const int64_t per = std::max(((int64_t)std::max(1, B) * ctx + kFillWorkgroups - 1) / kFillWorkgroups,
                               (ctx + kMaxSplitsForFill - 1) / kMaxSplitsForFill);
  return (int32_t)std::min<int64_t>(kChunk, std::max<int64_t>(kTile, (per + kTile - 1) / kTile * kTile));
}

int32_t decode_max_splits(int32_t B, int32_t max_context_len) {
  const int32_t c = decode_chunk_keys(B, max_context_len);
  return std::max<int32_t>(1, (max_context_len + c - 1) / c);
}

size_t decode_workspace_bytes(int32_t B, int32_t Hq, int32_t D, int32_t max_context_len) {
  return (size_t)4 * (size_t)B * (size_t)Hq * (size_t)decode_max_splits(B, max_context_len) *
         (size_t)(D + 2);
}

// HB: KV heads per workgroup (8 / HB waves share one head's key tiles).
template <int D, int G, int HB>
__global__ __launch_bounds__(512, 4) void attn_decode_split_kernel(
    const __bf16* __restrict__ q, int64_t q_stride, const __bf16* __restrict__ kc, const __bf16* __restrict__ vc,
    const int32_t* __restrict__ table, const int32_t* __restrict__ ctx, int Hq, int Hkv,
    int log2bs, int max_blocks, int64_t num_blocks, int max_splits, int chunk_keys, float scale_log2,
    float* __restrict__ ws_o, float* __restrict__ ws_ml) {
  constexpr int CPR = D / 8;             // 16-byte chunks per cache row
  constexpr int KSTEPS = D / 32;         // MFMA k-steps over the head dim (QK)
  constexpr int DT = D / 16;             // 16-wide output tiles over the head dim (PV)
  constexpr int WPH = kWaves / HB;       // waves sharing one head
  constexpr int VROWS = 64 / CPR;        // V rows per 1 KB wave load
  constexpr int VLOADS = kTile / VROWS;  // wave loads per V tile
  constexpr int VBYTES = kTile * D * 2;  // one V tile
  constexpr float kLazy = 8.f;
  __shared__ __attribute__((aligned(16))) char vbuf[kWaves][VBYTES];
  __shared__ int32_t pages[kMaxPages];

  const int split = blockIdx.x, hg = blockIdx.y, b = blockIdx.z;
  const int bs = 1 << log2bs;
  const int n = min(ctx[b], max_blocks << log2bs);
  const SplitPlan plan = plan_splits(n, max_splits, chunk_keys);
  const int k_begin = split * plan.chunk;
  if (split >= plan.splits || k_begin >= n) return;
  const int k_end = min(n, k_begin + plan.chunk);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int g = hg * HB + wave % HB;     // this wave's KV head
  const int wt = wave / HB;              // its share of the head's key tiles
  const int col = lane & 15, grp = lane >> 4;
  const int64_t row_elems = (int64_t)Hkv * D;
  OPS_LDS char* vb = (OPS_LDS char*)vbuf[wave];

  // Query heads of this group as the MFMA B operand (column = head).
  bf16x8 qf[KSTEPS];
  {
    const bool has = col < G;
    const __bf16* qrow = q + (int64_t)b * q_stride + ((int64_t)g * G + (has ? col : 0)) * D;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (has) w = *reinterpret_cast<const u32x4*>(qrow + s * 32 + grp * 8);
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // page ids of the current window (-1: not a valid block)
  const int32_t* trow = table + (int64_t)b * max_blocks;
  int p_first = 0, w_end = 0;
  auto load_pages = [&](int w0) {
    w_end = min(k_end, w0 + kChunk);
    p_first = w0 >> log2bs;
    const int p_count = ((w_end - 1) >> log2bs) - p_first + 1;
    for (int i = threadIdx.x; i < p_count; i += kWaves * 64) {
      const int blk = trow[p_first + i];
      pages[i] = (uint32_t)blk < (uint64_t)num_blocks ? blk : -1;
    }
  };
  // A key is used iff it lies in the window and its page is valid.
  auto key_ok = [&](int j) {
    return j < w_end && pages[(min(j, w_end - 1) >> log2bs) - p_first] >= 0;
  };
  // Cache row of key j for head g.  Skipped keys read the sequence's first
  // query row instead (finite data; their probability is exactly 0), so every
  // lane always issues every load and the vmcnt bookkeeping below is exact.
  const __bf16* dummy = q + (int64_t)b * q_stride;
  auto row_ptr = [&](const __bf16* cache, int j) -> const __bf16* {
    if (!key_ok(j)) return dummy;
    const int blk = pages[(j >> log2bs) - p_first];
    return cache + ((int64_t)blk * bs + (j & (bs - 1))) * row_elems + (int64_t)g * D;
  };

  // K of 32 keys in MFMA A-operand layout (registers, 2*KSTEPS loads); V of
  // the same keys DMA'd into this wave's LDS buffer (VLOADS loads).
  struct KRegs {
    u32x4 k[2][KSTEPS];
  };
  auto load_k = [&](int t0, KRegs& r) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const __bf16* kr = row_ptr(kc, t0 + sub * 16 + col);
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) r.k[sub][s] = *reinterpret_cast<const u32x4*>(kr + s * 32 + grp * 8);
    }
  };
  auto load_v = [&](int t0) {
#pragma unroll
    for (int i = 0; i < VLOADS; ++i) {
      const int row = i * VROWS + lane / CPR;
      const int c = (lane % CPR) ^ v_swz(row);  // logical chunk landing at this lane's slot
      global_load16_lds_nt(row_ptr(vc, t0 + row) + c * 8, vb + i * 1024);
    }
  };

  float m_run = -INFINITY, l_run = 0.f;  // softmax state of head `col` (lanes col < G)
  f32x4 acc[DT];                          // O[head 4*grp + r][d = 16*dt + col]
#pragma unroll
  for (int i = 0; i < DT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Scores, softmax and P V of one tile.
  auto compute_tile = [&](int t0, const KRegs& r) {
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
        const float sv = key_ok(j) ? st[sub][rr] * scale_log2 : -INFINITY;
        st[sub][rr] = sv;
        tmax = fmaxf(tmax, sv);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    // move the reference max only when the tile's max exceeds it by kLazy
    float alpha = 1.f;
    if (tmax > m_run + kLazy) {
      alpha = fast_exp2(m_run - tmax);
      m_run = tmax;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    // P as the MFMA A operand: slot e of lane (col, grp) is key 4*grp + e%4 + 16*(e/4)
    bf16x8 pa;
    float psum = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float p = fast_exp2(st[sub][rr] - m_use);
        psum += p;
        pa[sub * 4 + rr] = (__bf16)p;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    // rescale O rows (heads 4*grp + r) when any head's reference moved
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float a = __shfl(alpha, grp * 4 + rr, 64);
#pragma unroll
        for (int i = 0; i < DT; ++i) acc[i][rr] *= a;
      }
    }
    // V as the B operand: lane (d = 16*dt + col, group grp) needs keys
    // 4*grp + e (e < 4) and 16 + 4*grp + (e - 4); one transposed read each.
    const int trow0 = 4 * grp + (col >> 2);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int cc = dt * 16 + 4 * (col & 3);  // head-dim column of this lane's 8-byte chunk
      const int c16 = cc >> 3, half = (cc >> 2) & 1;
      const int r0 = trow0, r1 = trow0 + 16;
      const u32x2 lo = lds_read_tr16(vb + r0 * (D * 2) + ((c16 ^ v_swz(r0)) << 4) + half * 8);
      const u32x2 hi = lds_read_tr16(vb + r1 * (D * 2) + ((c16 ^ v_swz(r1)) << 4) + half * 8);
      const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
      acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vf, acc[dt], 0, 0, 0);
    }
  };

  // Each wave loads a tile, waits for it and uses it; latency is hidden by
  // the other waves of the CU (two workgroups of 8 waves fit: 64 KB of LDS
  // and at most 128 VGPRs each), not by register double buffering.  V is
  // refilled only after the previous tile's transposed reads fed its MFMAs.
  KRegs cur;
  for (int w0 = k_begin; w0 < k_end; w0 += kChunk) {
    if (w0 != k_begin) __syncthreads();  // every wave is done with the previous window
    load_pages(w0);
    __syncthreads();
    for (int t0 = w0 + wt * kTile; t0 < w_end; t0 += WPH * kTile) {
      load_k(t0, cur);
      load_v(t0);
      wait_vmem();
      compute_tile(t0, cur);
    }
  }

  // ---- merge the waves sharing a head (WPH > 1) through LDS, write partials
  // acc[dt][rr]: head 4*grp + rr, d = 16*dt + col.
  const int64_t slot_base = (int64_t)b * Hq * max_splits + split;
  if constexpr (WPH == 1) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int hh = 4 * grp + rr;
      if (hh < G) {
        const int64_t slot = slot_base + (int64_t)(g * G + hh) * max_splits;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) ws_o[slot * D + dt * 16 + col] = acc[dt][rr];
      }
    }
    if (col < G) {
      const int64_t slot = slot_base + (int64_t)(g * G + col) * max_splits;
      if (grp == 0) {
        ws_ml[slot * 2 + 0] = m_run;
        ws_ml[slot * 2 + 1] = l_run;
      }
    }
  } else {
    __syncthreads();  // the V buffers are reused for the merge
    float* red = reinterpret_cast<float*>(vbuf);  // [wave][G][D + 2]
    float* mine = red + wave * G * (D + 2);
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int hh = 4 * grp + rr;
      if (hh < G)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) mine[hh * (D + 2) + dt * 16 + col] = acc[dt][rr];
    }
    if (col < G && grp == 0) {
      mine[col * (D + 2) + D] = m_run;
      mine[col * (D + 2) + D + 1] = l_run;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < HB * G * D; idx += kWaves * 64) {
      const int hl = idx / (G * D), hh = (idx / D) % G, d = idx % D;  // head slot, query head, column
      float M = -INFINITY;
      for (int w = 0; w < WPH; ++w) M = fmaxf(M, red[((w * HB + hl) * G + hh) * (D + 2) + D]);
      float o = 0.f, l = 0.f;
      for (int w = 0; w < WPH; ++w) {
        const float* e = red + ((w * HB + hl) * G + hh) * (D + 2);
        const float f = e[D] == -INFINITY ? 0.f : fast_exp2(e[D] - M);
        o += f * e[d];
        l += f * e[D + 1];
      }
      const int64_t slot = slot_base + (int64_t)((hg * HB + hl) * G + hh) * max_splits;
      ws_o[slot * D + d] = o;
      if (d == 0) {
        ws_ml[slot * 2 + 0] = M;
        ws_ml[slot * 2 + 1] = l;
      }
    }
  }
}

// Merge the splits of one (sequence, head); one wave per pair.  The splits'
// maxima and weights are taken 64 at a time across the lanes; the weighted
// sum of their partial outputs then runs over the splits in order (lane l
// owns output columns l + 64 c), so the result is deterministic.
template <int D>
__global__ __launch_bounds__(64) void attn_decode_combine_kernel(
    const float* __restrict__ ws_o, const float* __restrict__ ws_ml, const int32_t* __restrict__ ctx,
    __bf16* __restrict__ o, int Hq, int log2bs, int max_blocks, int max_splits, int chunk_keys) {
  constexpr int DPL = D / 64;
  __shared__ float fw[64];
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int n = min(ctx[b], max_blocks << log2bs);
  const SplitPlan plan = plan_splits(n, max_splits, chunk_keys);
  const int64_t slot0 = ((int64_t)b * Hq + h) * max_splits;
  auto used = [&](int sp) { return sp < plan.splits && sp * plan.chunk < n; };
  float M = -INFINITY;
  for (int sp = lane; sp < plan.splits; sp += 64)
    if (used(sp)) M = fmaxf(M, ws_ml[(slot0 + sp) * 2]);
  M = wave_max(M);
  float acc[DPL] = {};
  float l = 0.f;
  for (int s0 = 0; s0 < plan.splits; s0 += 64) {
    float f = 0.f;
    const int sp = s0 + lane;
    if (used(sp)) {
      const float ms = ws_ml[(slot0 + sp) * 2];
      if (ms != -INFINITY) {  // -inf: every key of the split was skipped
        f = fast_exp2(ms - M);
        l += f * ws_ml[(slot0 + sp) * 2 + 1];
      }
    }
    fw[lane] = f;
    __builtin_amdgcn_wave_barrier();
    const int cnt = min(64, plan.splits - s0);
    // The rows of unused splits hold stale data: they are loaded anyway (so
    // that the loads do not wait on the weights) and dropped by the select.
    const float* base = ws_o + (slot0 + s0) * D + lane;
    int j = 0;
    for (; j + 8 <= cnt; j += 8) {
      float v[8][DPL];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int c = 0; c < DPL; ++c) v[u][c] = base[(j + u) * D + c * 64];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float fj = fw[j + u];
#pragma unroll
        for (int c = 0; c < DPL; ++c) acc[c] += fj == 0.f ? 0.f : fj * v[u][c];
      }
    }
    for (; j < cnt; ++j) {
      const float fj = fw[j];
#pragma unroll
      for (int c = 0; c < DPL; ++c) {
        const float v = base[j * D + c * 64];
        acc[c] += fj == 0.f ? 0.f : fj * v;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  l = wave_sum(l);
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int c = 0; c < DPL; ++c) o[((int64_t)b * Hq + h) * D + lane + c * 64] = (__bf16)(acc[c] * inv);
}

// ------------------------------------------------------------ fp32 path ----
template <int D>
__global__ __launch_bounds__(64) void attn_decode_f32_kernel(
    const float* __restrict__ q, int64_t q_stride, const float* __restrict__ kc, const float* __restrict__ vc,
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
  for (int d = lane; d < D; d += 64) qs[d] = q[(int64_t)b * q_stride + (int64_t)h * D + d];
  __syncthreads();
  float m_run = -INFINITY, l_run = 0.f, acc[DPL] = {};
  for (int kv0 = 0; kv0 < n; kv0 += 64) {
    const int j = kv0 + lane;
    float s = -INFINITY;  // keys in invalid pages are skipped
    int64_t row = -1;
    if (j < n) {
      const int blk = trow[j >> log2bs];
      if ((uint32_t)blk < (uint64_t)num_blocks) {
        row = (((int64_t)blk * bs + (j & (bs - 1))) * Hkv + g) * D;
        float dot = 0.f;
        for (int d = 0; d < D; ++d) dot = fmaf(qs[d], kc[row + d], dot);
        s = dot * scale;
      }
    }
    rows[lane] = row;
    const float m_new = fmaxf(m_run, wave_max(s));
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float p = row >= 0 ? expf(s - m_use) : 0.f;
    const float alpha = expf(m_run - m_use);
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

hipError_t launch_attn_decode(const void* q, int64_t q_stride, const void* kcache, const void* vcache,
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
                         static_cast<const float*>(q), q_stride, static_cast<const float*>(kcache),
                         static_cast<const float*>(vcache), table, ctx, static_cast<float*>(o), Hq,
                         Hkv, log2bs, max_blocks, num_blocks, scale);
    else
      hipLaunchKernelGGL((attn_decode_f32_kernel<64>), grid, dim3(64), 0, s,
                         static_cast<const float*>(q), q_stride, static_cast<const float*>(kcache),
                         static_cast<const float*>(vcache), table, ctx, static_cast<float*>(o), Hq,
                         Hkv, log2bs, max_blocks, num_blocks, scale);
    return hipGetLastError();
  }
  const int chunk_keys = decode_chunk_keys(B, max_context_len);
  const int max_splits = decode_max_splits(B, max_context_len);
  float* ws_o = static_cast<float*>(ws);
  float* ws_ml = ws_o + (size_t)B * Hq * max_splits * D;
  const float sl2 = scale * kLog2e;
  const int G = Hq / Hkv;
  const int HB = Hkv >= 8 ? 8 : Hkv;  // KV heads per workgroup (Hkv in {1, 2, 4} or a multiple of 8)
  const dim3 grid((unsigned)max_splits, (unsigned)(Hkv / HB), (unsigned)B);
#define OPS_DEC(DD, GG, HH)                                                                     \
  hipLaunchKernelGGL((attn_decode_split_kernel<DD, GG, HH>), grid, dim3(kWaves * 64), 0, s,     \
                     static_cast<const __bf16*>(q), q_stride, static_cast<const __bf16*>(kcache), \
                     static_cast<const __bf16*>(vcache), table, ctx, Hq, Hkv, log2bs, max_blocks, \
                     num_blocks, max_splits, chunk_keys, sl2, ws_o, ws_ml)
#define OPS_DEC_H(DD, GG)                    \
  switch (HB) {                              \
    case 1: OPS_DEC(DD, GG, 1); break;       \
    case 2: OPS_DEC(DD, GG, 2); break;       \
    case 4: OPS_DEC(DD, GG, 4); break;       \
    default: OPS_DEC(DD, GG, 8); break;      \
  }
#define OPS_DEC_G(DD)                   \
  switch (G) {                          \
    case 1: OPS_DEC_H(DD, 1) break;     \
    case 2: OPS_DEC_H(DD, 2) break;     \
    case 4: OPS_DEC_H(DD, 4) break;     \
    default: OPS_DEC_H(DD, 8) break;    \
  }
  if (D == 128) {
    OPS_DEC_G(128)
  } else {
    OPS_DEC_G(64)
  }
#undef OPS_DEC_G
#undef OPS_DEC_H
#undef OPS_DEC
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cgrid((unsigned)Hq, (unsigned)B);
  if (D == 128)
    hipLaunchKernelGGL((attn_decode_combine_kernel<128>), cgrid, dim3(64), 0, s, ws_o, ws_ml, ctx,
                       static_cast<__bf16*>(o), Hq, log2bs, max_blocks, max_splits, chunk_keys);
  else
    hipLaunchKernelGGL((attn_decode_combine_kernel<64>), cgrid, dim3(64), 0, s, ws_o, ws_ml, ctx,
                       static_cast<__bf16*>(o), Hq, log2bs, max_blocks, max_splits, chunk_keys);
  return hipGetLastError();
}

}  // namespace opscale
