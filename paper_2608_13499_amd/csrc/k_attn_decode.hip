// Decode attention: one new query token per sequence against its paged KV
// cache [num_blocks, block_size, Hkv, D].
//
// bf16 path, balanced split-KV.  The plan is the prefix sum (tcs) of the
// batch's 32-key tiles per sequence: up to 512 sequences every workgroup
// builds it in LDS from the context lengths (one lane a sequence), beyond that
// a one-workgroup plan kernel writes it, with each workgroup's first sequence,
// to the workspace.  A fixed grid of nwg workgroups (one per tile of B x
// max_context_len keys, at most 256 in all, one per CU, and 64 per sequence)
// takes equal consecutive ranges of the tile list, so every workgroup streams
// the same number of keys however ragged the contexts are, and a range may
// span sequence boundaries.
// Each (workgroup g, sequence b) segment of the range is processed on its own
// and leaves (max, sum, unnormalized output) in slot g + b of the caller's
// workspace: unique, as the ranges are ordered like the sequences.
// A workgroup of 8 waves owns one group of up to 8 KV heads: for the 8-head
// layer every wave takes one KV head and serves all G query heads of that
// head, so each page of the cache (block_size slots x all heads, contiguous)
// is streamed by one workgroup in one pass and each K/V row is read from HBM
// exactly once.
// Per 32 keys a wave does:
//   * scores S^T[key][head] = K Q^T on MFMA 16x16x32: A = 16 cached K rows
//     loaded straight from HBM into operand registers, B = the G query rows
//     zero-padded to 16 columns;
//   * online softmax per head in the log2 domain (lazy reference max);
//   * O[head][d] += P V on MFMA 16x16x32: the S^T accumulator is already the
//     A operand P (a lane holds one head and 8 keys), and V, DMA'd into LDS
//     row-major, is read as the B operand with ds_read_b64_tr_b16.
// A wave loads a tile and waits for it; the latency is covered by the other
// waves of the CU (one V buffer per wave: 64 KB of LDS, at most 128 VGPRs;
// the grid gives each CU one workgroup).  V is read with the nontemporal
// hint, the cache is streamed once.
// A second kernel merges the segments of a (sequence, head) in workgroup
// order, so the result is deterministic; for small batches it recomputes the
// sequence's tile range from the context lengths instead of reading the plan
// that another XCD just wrote.
//
// Keys whose page id is outside [0, num_blocks) are skipped.
//
// fp32 path: one wave per (sequence, head), exact expf, no workspace use.
#include <algorithm>
#include <cstdlib>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kTile = 32;    // keys per wave step
constexpr int kWaves = 8;    // waves per workgroup
constexpr int kChunk = 512;  // keys per page window
// Workgroups of a launch, at most (one per CU: the grid runs in one round,
// and 8 waves per CU keep fewer loads in flight, which streams HBM faster
// than 16 did); and per sequence of the batch, at most (so a sequence's merge
// takes about one 64-wide pass).
constexpr int kMaxWorkgroups = 256;
constexpr int kSeqWorkgroups = 64;
constexpr int kInlineB = kWaves * 64;  // up to this batch every workgroup builds the plan itself
// Page ids of one window of kChunk keys (any block size >= 1) fit in here.
constexpr int kMaxPages = kChunk + 1;

typedef short s16x4 __attribute__((ext_vector_type(4)));

// gfx950 transposed LDS read: within each 16-lane group, lane i receives
// element i % 4 of the 8-byte chunks addressed by lanes 4e + i / 4 (e = 0..3).
__device__ __forceinline__ u32x2 lds_read_tr16(const OPS_LDS char* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((OPS_LDS s16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// V rows in LDS: the 16-byte chunk c of row r sits at chunk c ^ v_swz(r).
// With this wave's lane-to-row mapping the transposed reads run as fast as a
// linear read (3.5 cycles per read on gfx950, measured) for an XOR with
// 2*(r mod 8) on 256-byte rows and with r mod 8 on 128-byte rows; 2*(r mod 4)
// took 4.
template <int D>
__device__ __forceinline__ int v_swz(int r) { return D == 128 ? (r & 7) << 1 : r & 7; }

// a value equal on every lane, moved to scalar registers
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
}  // namespace

// Workgroups per KV-head group of a launch with `groups` such groups: one per
// 32-key tile of the largest possible batch (B x max_context_len keys), at
// most kMaxWorkgroups in all and kSeqWorkgroups per sequence; each takes an
// equal share of the tiles that exist.
int32_t decode_workgroups(int32_t B, int32_t max_context_len, int32_t groups) {
  const int64_t b = std::max(1, B);
  const int64_t tiles = b * ((std::max(1, max_context_len) + kTile - 1) / kTile);
  const int64_t cap = std::max(1, kMaxWorkgroups / std::max(1, groups));
  return (int32_t)std::min<int64_t>(std::min<int64_t>(cap, tiles), b * kSeqWorkgroups);
}

namespace {
// Workspace: tile prefix sums tcs [B + 1] (int64), each workgroup's first
// sequence [nwg] (int32; large batches only), then the partial results of
// Hq heads x (nwg + B) slots, head-major (a head's slots are contiguous, as
// the merge reads them): outputs [.][D], then (max, sum) pairs.
struct DecodeWs {
  int64_t* tcs;
  int32_t* first;
  float *o, *ml;
  size_t bytes;
};
// nwg: the launch's workgroups per head group (at most those of one group,
// which size the workspace)
DecodeWs decode_ws(void* base, int32_t B, int32_t Hq, int32_t D, int32_t nwg) {
  const int64_t slots = (int64_t)nwg + B;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t tcs_bytes = up((size_t)(B + 1) * 8), first_bytes = B > kInlineB ? up((size_t)nwg * 4) : 0;
  char* p = static_cast<char*>(base);
  DecodeWs w{};
  w.tcs = reinterpret_cast<int64_t*>(p);
  w.first = p && first_bytes ? reinterpret_cast<int32_t*>(p + tcs_bytes) : nullptr;
  w.o = p ? reinterpret_cast<float*>(p + tcs_bytes + first_bytes) : nullptr;
  w.ml = w.o ? w.o + (size_t)slots * Hq * D : nullptr;
  w.bytes = tcs_bytes + first_bytes + (size_t)slots * Hq * (D + 2) * 4;
  return w;
}
}  // namespace

size_t decode_workspace_bytes(int32_t B, int32_t Hq, int32_t D, int32_t max_context_len) {
  return decode_ws(nullptr, B, Hq, D, decode_workgroups(B, max_context_len, 1)).bytes;
}

// HB: KV heads per workgroup (8 / HB waves share one head's key tiles).
// INL: B <= kInlineB, every workgroup builds the plan in LDS; else the plan
// kernel's tcs and first_b are read.
template <int D, int G, int HB, bool INL>
__global__ __launch_bounds__(512, 4) void attn_decode_split_kernel(
    const __bf16* __restrict__ q, int64_t q_stride, const __bf16* __restrict__ kc, const __bf16* __restrict__ vc,
    const int32_t* __restrict__ table, const int32_t* __restrict__ ctx, int Hq, int Hkv,
    int log2bs, int max_blocks, int64_t num_blocks, const int64_t* __restrict__ tcs,
    const int32_t* __restrict__ first_b, int B, int nwg,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_ml) {
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
  __shared__ int64_t tcs_s[INL ? kInlineB + 1 : 1];  // small batches: the plan, built here
  __shared__ int32_t n_s[INL ? kInlineB : 1];
  __shared__ uint32_t wsum[kWaves];

  const int wgi = blockIdx.x, hg = blockIdx.y;
  const int bs = 1 << log2bs;
  const int max_keys = max_blocks << log2bs;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if constexpr (INL) {
    // tcs_s[b] = tiles of sequences 0 .. b-1: a lane per sequence, a scan
    // within each wave (at most 64 x 2^26 tiles: fits 32 bits), then across
    const int t = threadIdx.x;
    const int n = t < B ? min(max(ctx[t], 0), max_keys) : 0;
    const uint32_t tiles = (uint32_t)(n + kTile - 1) / kTile;
    uint32_t x = tiles;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int64_t incl = x;
    for (int w = 0; w < wave; ++w) incl += wsum[w];
    if (t < B) {
      tcs_s[t] = incl - tiles;
      n_s[t] = n;
    }
    if (t == kWaves * 64 - 1) tcs_s[B] = incl;
    __syncthreads();
  }
  auto TC = [&](int i) -> int64_t {
    if constexpr (INL) return uniform64(tcs_s[i]);
    else return uniform64(tcs[i]);
  };
  // this workgroup's tiles [t_lo, t_hi) of the batch's tile list
  const int64_t t_total = TC(B);
  const int64_t t_lo = (int64_t)wgi * t_total / nwg, t_hi = (int64_t)(wgi + 1) * t_total / nwg;
  if (t_lo >= t_hi) return;

  const int g = hg * HB + wave % HB;     // this wave's KV head
  const int wt = wave / HB;              // its share of the head's key tiles
  const int col = lane & 15, grp = lane >> 4;
  const int64_t row_elems = (int64_t)Hkv * D;
  OPS_LDS char* vb = (OPS_LDS char*)vbuf[wave];

  // One segment: keys [k_begin, k_end) of sequence b, partial results to
  // slot pslot (wgi + b).
  auto segment = [&](const int b, const int k_begin, const int k_end, const int64_t pslot) {
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
      const int c = (lane % CPR) ^ v_swz<D>(row);  // logical chunk landing at this lane's slot
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
      const u32x2 lo = lds_read_tr16(vb + r0 * (D * 2) + ((c16 ^ v_swz<D>(r0)) << 4) + half * 8);
      const u32x2 hi = lds_read_tr16(vb + r1 * (D * 2) + ((c16 ^ v_swz<D>(r1)) << 4) + half * 8);
      const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
      acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vf, acc[dt], 0, 0, 0);
    }
  };

  // Each wave loads a tile, waits for it and uses it; latency is hidden by
  // the other 7 waves of the CU, not by register double buffering.  V is
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
  // head-major partials: entry (head, slot) at head * (nwg + B) + slot
  const int64_t nslots = (int64_t)nwg + B;
  if constexpr (WPH == 1) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int hh = 4 * grp + rr;
      if (hh < G) {
        const int64_t slot = (int64_t)(g * G + hh) * nslots + pslot;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) ws_o[slot * D + dt * 16 + col] = acc[dt][rr];
      }
    }
    if (col < G) {
      const int64_t slot = (int64_t)(g * G + col) * nslots + pslot;
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
      const int64_t slot = (int64_t)((hg * HB + hl) * G + hh) * nslots + pslot;
      ws_o[slot * D + d] = o;
      if (d == 0) {
        ws_ml[slot * 2 + 0] = M;
        ws_ml[slot * 2 + 1] = l;
      }
    }
  }
  };  // segment

  // the sequences this workgroup's tiles belong to, in order; the first:
  // small batches bisect the plan in LDS (largest b with tcs[b] <= t_lo),
  // large ones take it from the plan kernel
  int b_first;
  if constexpr (INL) {
    int lo = 0, hi = B;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (tcs_s[mid] <= t_lo) lo = mid;
      else hi = mid;
    }
    b_first = __builtin_amdgcn_readfirstlane(lo);
  } else {
    b_first = __builtin_amdgcn_readfirstlane(first_b[wgi]);
  }
  bool first = true;
  for (int b = b_first; b < B; ++b) {
    const int64_t tb = TC(b);
    if (tb >= t_hi) break;
    const int64_t s0 = max(t_lo, tb), s1 = min(t_hi, TC(b + 1));
    if (s0 >= s1) continue;  // a sequence without keys
    int n;
    if constexpr (INL) n = __builtin_amdgcn_readfirstlane(n_s[b]);
    else n = __builtin_amdgcn_readfirstlane(min(ctx[b], max_keys));
    if (!first) __syncthreads();  // every wave is done with the previous segment's LDS
    first = false;
    segment(b, (int)(s0 - tb) * kTile, min(n, (int)(s1 - tb) * kTile), (int64_t)wgi + b);
  }
}

// Plan of a large batch (one workgroup): tcs[b] = tiles (kTile keys) of
// sequences 0 .. b-1, n clamped to the block table, tcs[B] the batch's total;
// then first_b[g] = the sequence holding the first tile of workgroup g (tile
// floor(g T / nwg)), written by the sequence that holds it.
__global__ __launch_bounds__(1024) void attn_decode_plan_kernel(const int32_t* __restrict__ ctx, int B,
                                                                int max_keys, int nwg, int64_t* __restrict__ tcs,
                                                                int32_t* __restrict__ first_b) {
  __shared__ int64_t part[1024];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  auto tiles_of = [&](int b) { return (min(max(ctx[b], 0), max_keys) + kTile - 1) / kTile; };
  for (int b0 = 0; b0 < B; b0 += 1024) {
    const int b = b0 + threadIdx.x;
    const int nt = b < B ? tiles_of(b) : 0;
    part[threadIdx.x] = nt;
    __syncthreads();
    // inclusive scan (Hillis-Steele) over the 1024 entries
    for (int o = 1; o < 1024; o <<= 1) {
      const int64_t v = threadIdx.x >= o ? part[threadIdx.x - o] : 0;
      __syncthreads();
      part[threadIdx.x] += v;
      __syncthreads();
    }
    const int64_t c = carry;
    if (b < B) tcs[b] = c + part[threadIdx.x] - nt;
    __syncthreads();
    if (threadIdx.x == 1023) carry = c + part[1023];
    __syncthreads();
  }
  const int64_t T = carry;
  if (threadIdx.x == 0) tcs[B] = T;
  if (T == 0) return;
  // workgroups g with floor(g T / nwg) in [lo, hi): g in [ceil(lo nwg / T), ceil(hi nwg / T))
  for (int b = threadIdx.x; b < B; b += 1024) {
    const int64_t lo = tcs[b], hi = lo + tiles_of(b);  // tcs[b]: this thread's own store
    const int64_t g1 = (hi * nwg + T - 1) / T;
    for (int64_t g = (lo * nwg + T - 1) / T; g < g1; ++g) first_b[g] = b;
  }
}

// Merge the partial results of one (sequence, head); one wave per pair.  The
// sequence's tiles [tcs[b], tcs[b + 1]) were processed by workgroups g0 .. g1
// (workgroup g holds tiles [g T / nwg, (g + 1) T / nwg)), whose partials sit
// in slots g + b.  Their maxima and weights are taken 64 at a time across the
// lanes; the weighted sum then runs over them in order (lane l owns output
// columns l + 64 c), so the result is deterministic.
// INL (B <= kInlineB): the sequence's tile range and the batch total are
// recomputed from the context lengths (read-only, already cached by the split
// kernel's loads) rather than read from the plan.
template <int D, bool INL>
__global__ __launch_bounds__(64) void attn_decode_combine_kernel(
    const float* __restrict__ ws_o, const float2* __restrict__ ws_ml, const int64_t* __restrict__ tcs,
    const int32_t* __restrict__ ctx, int max_keys, __bf16* __restrict__ o, int Hq, int B, int nwg) {
  constexpr int DPL = D / 64;
  __shared__ float fw[64];
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  __bf16* orow = o + ((int64_t)b * Hq + h) * D;
  auto tiles_of = [&](int c) { return (min(max(c, 0), max_keys) + kTile - 1) / kTile; };
  int64_t T, ft, lt;
  if constexpr (INL) {
    int c[kInlineB / 64];  // unconditional (clamped) loads, all issued before the first use
#pragma unroll
    for (int k = 0; k < kInlineB / 64; ++k) c[k] = ctx[min(lane + 64 * k, B - 1)];
    int pre = 0, all = 0;  // at most 8 sequences of < 2^26 tiles a lane
#pragma unroll
    for (int k = 0; k < kInlineB / 64; ++k) {
      const int t = lane + 64 * k < B ? tiles_of(c[k]) : 0;
      all += t;
      pre += lane + 64 * k < b ? t : 0;
    }
    // wave sums of up to 2^35 in two 32-bit halves
    auto sum = [](int v) { return ((int64_t)wave_sum_i(v >> 16) << 16) + wave_sum_i(v & 0xffff); };
    ft = sum(pre);
    T = sum(all);
    lt = ft + tiles_of(ctx[b]) - 1;
  } else {
    T = tcs[B];
    ft = tcs[b];
    lt = tcs[b + 1] - 1;
  }
  if (lt < ft) {  // no keys: a zero row
#pragma unroll
    for (int c = 0; c < DPL; ++c) orow[lane + c * 64] = (__bf16)0.f;
    return;
  }
  // first / last workgroup: g(t) = floor(((t + 1) nwg - 1) / T); 32-bit
  // while the products fit
  int g0, g1;
  const bool small = T < (1 << 21);  // nwg <= 512: products < 2^30
  if (small) {
    const int t32 = (int)T;
    g0 = ((int)(ft + 1) * nwg - 1) / t32;
    g1 = ((int)(lt + 1) * nwg - 1) / t32;
  } else {
    g0 = (int)(((ft + 1) * nwg - 1) / T);
    g1 = (int)(((lt + 1) * nwg - 1) / T);
  }
  const int S = g1 - g0 + 1;
  // head-major partials: this head's slots g0 + b .. g1 + b are contiguous
  const int64_t base = (int64_t)h * ((int64_t)nwg + B) + g0 + b;
  auto slot = [&](int s_) { return base + s_; };
  // workgroups with an empty tile range (only if T < nwg) wrote nothing;
  // every other one in [g0, g1] holds a segment of this sequence
  auto live = [&](int s_) {
    if (T >= nwg) return true;
    const int gg = g0 + s_, t32 = (int)T;
    return gg * t32 / nwg < (gg + 1) * t32 / nwg;
  };
  auto ml_at = [&](int sp) {
    return sp < S && live(sp) ? ws_ml[slot(sp)] : float2{-INFINITY, 0.f};
  };
  const float2 ml0 = ml_at(lane);  // the first 64 partials' (max, sum) stay in registers
  float M = ml0.x;
  for (int sp = lane + 64; sp < S; sp += 64) M = fmaxf(M, ml_at(sp).x);
  M = wave_max_f(M);
  float acc[DPL] = {};
  float l = 0.f;
  for (int s0 = 0; s0 < S; s0 += 64) {
    const float2 e = s0 == 0 ? ml0 : ml_at(s0 + lane);
    float f = 0.f;
    if (e.x != -INFINITY) {  // -inf: no segment, or every key of it was skipped
      f = fast_exp2(e.x - M);
      l += f * e.y;
    }
    fw[lane] = f;
    __builtin_amdgcn_wave_barrier();
    const int cnt = min(64, S - s0);
    // the partials' rows are loaded 8 at a time without waiting on the
    // weights; rows of dead slots are dropped by the select
    int j = 0;
    for (; j + 8 <= cnt; j += 8) {
      float v[8][DPL];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int c = 0; c < DPL; ++c) v[u][c] = ws_o[slot(s0 + j + u) * D + lane + c * 64];
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
        const float v = ws_o[slot(s0 + j) * D + lane + c * 64];
        acc[c] += fj == 0.f ? 0.f : fj * v;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  l = wave_sum_f(l);
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int c = 0; c < DPL; ++c) orow[lane + c * 64] = (__bf16)(acc[c] * inv);
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
  const int HB = Hkv >= 8 ? 8 : Hkv;  // KV heads per workgroup (Hkv in {1, 2, 4} or a multiple of 8)
  const int nwg = decode_workgroups(B, max_context_len, Hkv / HB);
  const DecodeWs w = decode_ws(ws, B, Hq, D, nwg);
  float* ws_o = w.o;
  float* ws_ml = w.ml;
  if (B > kInlineB) {
    hipLaunchKernelGGL(attn_decode_plan_kernel, dim3(1), dim3(1024), 0, s, ctx, B, max_blocks << log2bs, nwg,
                       w.tcs, w.first);
    const hipError_t e0 = hipGetLastError();
    if (e0 != hipSuccess) return e0;
  }
  const float sl2 = scale * kLog2e;
  const int G = Hq / Hkv;
  const dim3 grid((unsigned)nwg, (unsigned)(Hkv / HB));
#define OPS_DEC(DD, GG, HH)                                                                      \
  if (B <= kInlineB)                                                                             \
    OPS_DEC_L(DD, GG, HH, true);                                                                 \
  else                                                                                           \
    OPS_DEC_L(DD, GG, HH, false)
#define OPS_DEC_L(DD, GG, HH, II)                                                                   \
  hipLaunchKernelGGL((attn_decode_split_kernel<DD, GG, HH, II>), grid, dim3(kWaves * 64), 0, s,     \
                     static_cast<const __bf16*>(q), q_stride, static_cast<const __bf16*>(kcache), \
                     static_cast<const __bf16*>(vcache), table, ctx, Hq, Hkv, log2bs, max_blocks, \
                     num_blocks, w.tcs, w.first, B, nwg, sl2, ws_o, ws_ml)
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
#undef OPS_DEC_L
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cgrid((unsigned)Hq, (unsigned)B);
  const int max_keys = max_blocks << log2bs;
  __bf16* ob = static_cast<__bf16*>(o);
#define OPS_COMB(DD, II)                                                                                  \
  hipLaunchKernelGGL((attn_decode_combine_kernel<DD, II>), cgrid, dim3(64), 0, s, ws_o,                  \
                     reinterpret_cast<const float2*>(ws_ml), w.tcs, ctx,                                    \
                     max_keys, ob, Hq, B, nwg)
  if (D == 128) {
    if (B <= kInlineB) OPS_COMB(128, true);
    else OPS_COMB(128, false);
  } else {
    if (B <= kInlineB) OPS_COMB(64, true);
    else OPS_COMB(64, false);
  }
#undef OPS_COMB
  return hipGetLastError();
}

}  // namespace opscale
