// Causal grouped-query prefill attention over a ragged batch of prompts.
//
// bf16 path (D = 64 or 128): one workgroup of 4 waves per (prompt, KV head,
// query tile).  The waves are the query heads of one GQA group (up to 4) times
// query sub-tiles of 32 rows, so every K/V tile staged in LDS is shared by all
// the heads that read it.  Per 64-key K/V tile a wave computes the transposed
// score tile S^T = K Q^T on MFMA 32x32x16 (A = K rows from LDS, B = its 32
// query rows held in registers), so each lane owns one query and 16 keys per
// 32-key block: the online-softmax row max needs one cross-lane step.  The
// probabilities P^T, rounded to bf16, are then directly the B operand of
// O^T += V^T P^T, with V^T staged transposed in LDS; O^T keeps one query per
// lane too, so the softmax rescale is a per-lane scalar.
//
// The contraction index of an MFMA is summed over, so any bijection between
// the instruction's k slots and the keys of a 16-key step is valid as long as
// both operands use it.  Here slot e of lane half h in step s is key
// 16s + 8(e/4) + 4h + e%4: exactly the keys the S^T accumulator leaves in that
// lane, so P needs no shuffle.
//
// Launch: grid.x = (prompt, KV head, head block), grid.y = query-tile level,
// highest level first, so the most expensive tiles (the ends of the longest
// prompts, which see the most keys) start earliest.  A block whose level is
// beyond its prompt exits at once; levels past gridDim.y are looped, so the
// result never depends on max_seqlen.
//
// fp32 path: one wave per (token, head), keys 64 at a time, exact expf; it
// serves the fp32 parity configuration.
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBKV = 64;  // keys per K/V tile
}  // namespace

template <int D>
struct PrefillSmem {
  // One stage holds a 64-key K tile and a 64-key V tile, both row-major (D
  // bf16 per row) and both filled by buffer_load ... lds.  The 16-byte chunk c
  // of K row r sits at chunk c ^ k_swz(r); of V row r at chunk c ^ v_swz(r).
  static constexpr int kRowBytes = D * 2;
  static constexpr int kTileBytes = kBKV * kRowBytes;
  static constexpr int kStage = 2 * kTileBytes;
  static constexpr int kTotal = 2 * kStage;
};

// K is read as the MFMA A operand: 32 consecutive rows at one chunk.  Any 8
// (and 16) consecutive rows must hit distinct 16-byte bank groups.
template <int D>
__device__ __forceinline__ int k_swz(int r) {
  return D == 128 ? (r & 15) : ((r ^ (r >> 3)) & 7);
}
// V is read with ds_read_b64_tr_b16: a 16-lane group reads 4 consecutive rows
// x 32 bytes (two 16-byte chunks).  XOR-ing the chunk with 4*(r mod 4) for
// 256-byte rows, 2*(r mod 4) for 128-byte rows, makes these reads as fast as
// a linear one (3.5 cycles per read on gfx950, measured; 2*(r mod 4) on
// 256-byte rows takes 4).
template <int D>
__device__ __forceinline__ int v_swz(int r) { return D == 128 ? (r & 3) << 2 : (r & 3) << 1; }

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Transposed LDS read (gfx950 ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane i receives element i % 4 of the 8-byte chunks addressed by
// lanes 4e + i / 4 of its group, for e = 0..3.
__device__ __forceinline__ u32x2 lds_read_tr16(const OPS_LDS char* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((OPS_LDS s16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// The value lane i ^ 32 holds (v_permlane32_swap: no LDS round trip).
__device__ __forceinline__ float other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  // lanes 0-31: r[1] holds lanes 32-63; lanes 32-63: r[0] holds lanes 0-31
  return __uint_as_float((__lane_id() < 32) ? r[1] : r[0]);
}

// 16 bytes per lane from a buffer into LDS at lds_wave_base + lane * 16
// (buffer_load_dwordx4 ... lds, the LDS base in M0), written as assembly so
// that the compiler does not track it.  Tracked, it makes the first V read of
// every step wait for all loads in flight (it cannot tell that they fill the
// other stage), so the next tile's loads would never overlap P V.  The
// kernel orders these loads itself: wait_vmem() and a barrier before any
// wave reads a stage they fill, and a barrier before a stage is refilled.
__device__ __forceinline__ void lds_dma16(uint64_t base, uint32_t nrec, OPS_LDS char* lds_wave_base,
                                          uint32_t voff) {
  const u32x4 rs = {(uint32_t)base, (uint32_t)(base >> 32) & 0xffffu, nrec, (uint32_t)kBufferFlags};
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_wave_base);
  // s_nop 4: the compiler's hazard check does not see into the assembly, so
  // the wait states it would insert come first: an LDS DMA reading M0 right
  // after M0 is written (one), and a buffer instruction reading an SGPR of its
  // descriptor that a VALU instruction (v_readfirstlane) wrote (five, gfx9)
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "{m0}"(m0v), "v"(voff), "s"(rs));
}

// Prompts the work-list schedule can hold in LDS (more use the grid schedule).
constexpr int kMaxListB = 1024;

// Two schedules over the same tiles (a tile: one prompt, one KV head, one
// head block, one query-tile level), each tile computed the same way, so the
// output does not depend on the schedule:
//  * grid (LIST = false): blockIdx = (prompt x KV head x head block, level),
//    highest level first; workgroups whose prompt has no tile at their level
//    return at once.
//  * work list (LIST = true): workgroup i takes item i of the level-major list
//    of the tiles that exist (highest level first, then prompt, KV head and
//    head block), so no workgroup is launched for a missing tile.
template <int D, bool LIST>
__global__ __launch_bounds__(256, 2) void attn_prefill_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    int64_t q_stride, int64_t kv_stride, __bf16* __restrict__ o, const int32_t* __restrict__ cu,
    int B, int Hq, int Hkv, int hpb, float scale_log2, int causal) {
  using S = PrefillSmem<D>;
  constexpr int CPR = D / 8;          // 16-byte chunks per row
  constexpr int DSTEPS = D / 16;      // MFMA k-steps over the head dim
  constexpr int DT = D / 32;          // 32-wide output tiles over the head dim
  // Lazy rescaling: the running max only moves when a tile's max exceeds it by
  // more than this (log2 units), so probabilities stay <= 2^kLazy and the
  // output rescale is skipped on most tiles.  Exact: numerator and
  // denominator use the same reference.
  constexpr float kLazy = 8.f;
  __shared__ __attribute__((aligned(16))) char smem_raw[S::kTotal];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;

  const int G = Hq / Hkv;
  const int nhb = G / hpb;
  const int qsub = 4 / hpb;
  const int BQ = 32 * qsub;
  const int bq_shift = 5 + __builtin_ctz(qsub);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int qs = wave / hpb;
  const int fr = lane & 31, fh = lane >> 5;
  // lane roles in the transposed V reads: 16-lane group tg, member tc
  const int tg = lane >> 4, tc = lane & 15;
  const int tr_key = 4 * (tg >> 1) + (tc >> 2);               // + 16 s (+ 8 for the upper half)
  const int tr_col = 16 * (tg & 1) + 4 * (tc & 3);            // + 32 dt

  // One query tile: prompt b, KV head g, head block hb, level t.
  auto do_tile = [&](const int b, const int g, const int hb, const int t, const int seq0, const int L) {
    const int h = g * G + hb * hpb + wave % hpb;
    const int q_lo = t * BQ + qs * 32;          // first query of this wave
    const int q_pos = q_lo + fr;                 // this lane's query
    const int blk_q_hi = min(L, (t + 1) * BQ);   // one past the block's last query
    const int kv_end = causal ? blk_q_hi : L;
    const int nkv = (kv_end + kBKV - 1) / kBKV;

    // This wave's 32 query rows as MFMA B operand: chunk 2*s + fh of row q_pos.
    bf16x8 qf[DSTEPS];
    {
      // (the record count is wave-uniform; readfirstlane keeps the
      // descriptor in scalar registers)
      const int rows = max(0, min(32, L - q_lo));
      const uint32_t nrec = __builtin_amdgcn_readfirstlane(
          rows > 0 ? (uint32_t)(((int64_t)(rows - 1) * q_stride + D) * 2) : 0u);
      const __amdgpu_buffer_rsrc_t qr = make_rsrc(q + (int64_t)(seq0 + q_lo) * q_stride + (int64_t)h * D, nrec);
#pragma unroll
      for (int s = 0; s < DSTEPS; ++s) {
        const u32x4 w = buffer_load16(qr, (uint32_t)(((int64_t)fr * q_stride + (2 * s + fh) * 8) * 2));
        qf[s] = __builtin_bit_cast(bf16x8, w);
      }
    }

    f32x16 acc[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) acc[i] = f32x16{};
    float m_run = -INFINITY, l_part = 0.f;  // running max (log2 units) and partial sum

    // K and V tiles: LDS DMA, rows past the prompt read as zeros.
    auto load_kv = [&](int kv0, int stage) {
      const int rows = min(kBKV, L - kv0);
      const uint32_t nrec = __builtin_amdgcn_readfirstlane((uint32_t)(((int64_t)(rows - 1) * kv_stride + D) * 2));
      const int64_t off = (int64_t)(seq0 + kv0) * kv_stride + (int64_t)g * D;
      const uint64_t kb = (uint64_t)(uintptr_t)(k + off), vb = (uint64_t)(uintptr_t)(v + off);
      OPS_LDS char* dk = smem + stage * S::kStage;
      OPS_LDS char* dv = dk + S::kTileBytes;
      constexpr int ROWS_PER_LOAD = 64 / CPR;  // rows covered by one 1 KB wave load
      constexpr int LOADS = kBKV / ROWS_PER_LOAD / 4;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const int grp = i * 4 + wave;
        const int r = grp * ROWS_PER_LOAD + lane / CPR;
        const int pc = lane % CPR;
        lds_dma16(kb, nrec, dk + grp * 1024, (uint32_t)(((int64_t)r * kv_stride + (pc ^ k_swz<D>(r)) * 8) * 2));
        lds_dma16(vb, nrec, dv + grp * 1024, (uint32_t)(((int64_t)r * kv_stride + (pc ^ v_swz<D>(r)) * 8) * 2));
      }
    };

    if (nkv > 0) load_kv(0, 0);
    for (int it = 0; it < nkv; ++it) {
      const int kv0 = it * kBKV;
      wait_vmem();
      __syncthreads();
      if (it + 1 < nkv) load_kv(kv0 + kBKV, (it + 1) & 1);
      const OPS_LDS char* ks = smem + (it & 1) * S::kStage;
      const OPS_LDS char* vs = ks + S::kTileBytes;
      // Skip tiles that are entirely in this wave's causal future.
      const bool active = !(causal && kv0 > q_lo + 31) && q_lo < L;
      if (!active) continue;
      f32x16 st[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        st[kb] = f32x16{};
        const int r = kb * 32 + fr;
#pragma unroll
        for (int s = 0; s < DSTEPS; ++s) {
          const int c = 2 * s + fh;
          const bf16x8 kf = *reinterpret_cast<const OPS_LDS bf16x8*>(
              ks + r * S::kRowBytes + ((c ^ k_swz<D>(r)) << 4));
          st[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], st[kb], 0, 0, 0);
        }
      }
      // mask (only tiles that reach past the diagonal or the prompt end):
      // key kv0 + fh*4 + off is visible iff off <= lim, off a constant per element
      if ((causal && kv0 + kBKV - 1 > q_lo) || kv0 + kBKV > L) {
        const int lim = (causal ? min(q_pos, L - 1) : L - 1) - kv0 - fh * 4;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kb * 32 + (e >> 2) * 8 + (e & 3) > lim) st[kb][e] = -INFINITY;
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, st[kb][e]);
      tmax = fmaxf(tmax, other_half(tmax)) * scale_log2;
      // move the reference max only when the tile's max exceeds it by kLazy
      if (tmax > m_run + kLazy) {
        const float alpha = fast_exp2(m_run - tmax);  // 0 on the first tile
        l_part *= alpha;
#pragma unroll
        for (int i = 0; i < DT; ++i) acc[i] *= alpha;
        m_run = tmax;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float psum = 0.f;
      bf16x8 pf[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = fast_exp2(fmaf(st[kb][e], scale_log2, -m_use));
          psum += p;
          pf[kb * 2 + (e >> 3)][e & 7] = (__bf16)p;
        }
      l_part += psum;
      // O^T[d][i] += sum_key V^T[d][key] P^T[key][i]; the A operand (V^T, lane:
      // d = 32 dt + fr, keys 16 s + 8 (e/4) + 4 fh + e%4) comes from two
      // transposed reads of the row-major V tile.
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int r0 = 16 * s + tr_key, r1 = r0 + 8;
          const int cc = 32 * dt + tr_col;  // head-dim column of this lane's 8-byte chunk
          const int c16 = cc >> 3, half = (cc >> 2) & 1;
          const u32x2 lo = lds_read_tr16(vs + r0 * S::kRowBytes + ((c16 ^ v_swz<D>(r0)) << 4) + half * 8);
          const u32x2 hi = lds_read_tr16(vs + r1 * S::kRowBytes + ((c16 ^ v_swz<D>(r1)) << 4) + half * 8);
          const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
          acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[s], acc[dt], 0, 0, 0);
        }
      }
    }

    // normalize and store: lane owns query q_pos; acc[dt][e] is
    // d = dt*32 + (e/4)*8 + fh*4 + e%4.
    const float l_tot = l_part + other_half(l_part);
    if (q_pos < L && q_lo < L) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      __bf16* orow = o + ((int64_t)(seq0 + q_pos) * Hq + h) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          u32x2 out;
          out[0] = pack_bf2(acc[dt][gq * 4 + 0] * inv, acc[dt][gq * 4 + 1] * inv);
          out[1] = pack_bf2(acc[dt][gq * 4 + 2] * inv, acc[dt][gq * 4 + 3] * inv);
          *reinterpret_cast<u32x2*>(orow + dt * 32 + gq * 8 + fh * 4) = out;
        }
    }
    wait_vmem();      // (a stage load of a wave with no active step may still be in flight)
    __syncthreads();  // the next tile reuses the LDS stages
  };

  if constexpr (!LIST) {
    const int bx = blockIdx.x;
    const int b = bx / (Hkv * nhb);
    const int g = (bx / nhb) % Hkv;
    const int hb = bx % nhb;
    const int seq0 = cu[b];
    const int L = cu[b + 1] - seq0;
    const int ntiles = (L + BQ - 1) / BQ;
    for (int t = gridDim.y - 1 - blockIdx.y; t < ntiles; t += gridDim.y) do_tile(b, g, hb, t, seq0, L);
  } else {
    // n_s[b]: query tiles of prompt b.  The list holds, for every level t from
    // the highest down, the prompts with a tile at level t (batch order), each
    // with its HG (KV head, head block) pairs.  The tile groups at levels >= t
    // number F(t) = sum_b max(0, n_b - t), so item group q sits at the level
    // t with F(t + 1) <= q < F(t), found by bisection.
    // The table (cu_s, n_s) sits in the K/V stage buffers, so it is rebuilt
    // for every item: the tile's loads overwrite it.
    static_assert((2 * kMaxListB + 1) * 4 <= S::kTotal, "work table does not fit the stage buffers");
    OPS_LDS int32_t* cu_s = (OPS_LDS int32_t*)smem;
    OPS_LDS int32_t* n_s = cu_s + kMaxListB + 1;
    const int HG = Hkv * nhb;
    for (int64_t i = blockIdx.x;; i += gridDim.x) {
      for (int x = threadIdx.x; x <= B; x += 256) {
        const int c = cu[x];
        cu_s[x] = c;
        if (x < B) n_s[x] = (cu[x + 1] - c + BQ - 1) >> bq_shift;
      }
      __syncthreads();
      // (values below are equal in every lane and every wave; the first 64
      // tile counts stay in a register)
      const int n0 = lane < B ? n_s[lane] : 0;
      auto F = [&](int t) {
        int acc_n = max(0, n0 - t);
        for (int b0 = 64; b0 < B; b0 += 64)
          if (b0 + lane < B) acc_n += max(0, n_s[b0 + lane] - t);
        return wave_sum_i(acc_n);
      };
      int top = n0;
      for (int b0 = 64; b0 < B; b0 += 64)
        if (b0 + lane < B) top = max(top, n_s[b0 + lane]);
      top = wave_max_i(top);
      if (i >= (int64_t)F(0) * HG) break;
      const int qg = (int)(i / HG), r = (int)(i % HG);
      int lo = 0, hi = top;  // F(lo) > qg >= F(hi)
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (F(mid) > qg) lo = mid;
        else hi = mid;
      }
      const int t = lo;
      // the j-th prompt (batch order) with a tile at level t
      int j = qg - F(t + 1);
      int b = 0;
      for (int b0 = 0; b0 < B; b0 += 64) {
        const bool has = b0 == 0 ? n0 > t : (b0 + lane < B && n_s[b0 + lane] > t);
        const uint64_t m = __builtin_amdgcn_ballot_w64(has);
        const int pc = __builtin_popcountll(m);
        if (j < pc) {
          const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
          b = b0 + __builtin_ctzll(__builtin_amdgcn_ballot_w64(has && before == j));
          break;
        }
        j -= pc;
      }
      // the values are uniform; saying so keeps the tile's buffer descriptors
      // in scalar registers
      const int ub = __builtin_amdgcn_readfirstlane(b);
      const int s0 = __builtin_amdgcn_readfirstlane(cu_s[ub]);
      const int s1 = __builtin_amdgcn_readfirstlane(cu_s[ub + 1]);
      __syncthreads();  // every wave has read the table
      do_tile(ub, r / nhb, r % nhb, t, s0, s1 - s0);
    }
  }
}

// ------------------------------------------------------------ fp32 path ----
// One wave per (token, query head).  Lane j scores key kv0 + j; probabilities
// go through LDS and each lane accumulates D/64 output columns.
template <int D>
__global__ __launch_bounds__(64) void attn_prefill_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    int64_t q_stride, int64_t kv_stride, float* __restrict__ o, const int32_t* __restrict__ cu,
    int B, int Hq, int Hkv, float scale, int causal) {
  constexpr int DPL = D / 64;
  __shared__ float qs[D];
  __shared__ float ps[64];
  const int t = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  // prompt of token t
  int lo = 0, hi = B;  // cu[lo] <= t < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid;
  }
  const int seq0 = cu[lo], L = cu[lo + 1] - seq0, i = t - seq0;
  const int g = h / (Hq / Hkv);
  for (int d = lane; d < D; d += 64) qs[d] = q[(int64_t)t * q_stride + (int64_t)h * D + d];
  __syncthreads();
  const int kv_end = causal ? i + 1 : L;
  float m_run = -INFINITY, l_run = 0.f, acc[DPL] = {};
  for (int kv0 = 0; kv0 < kv_end; kv0 += 64) {
    const int j = kv0 + lane;
    float s = -INFINITY;
    if (j < kv_end) {
      const float* kr = k + (int64_t)(seq0 + j) * kv_stride + (int64_t)g * D;
      float dot = 0.f;
      for (int d = 0; d < D; ++d) dot = fmaf(qs[d], kr[d], dot);
      s = dot * scale;
    }
    const float m_new = fmaxf(m_run, wave_max(s));
    const float p = j < kv_end ? expf(s - m_new) : 0.f;
    const float alpha = expf(m_run - m_new);
    l_run = l_run * alpha + wave_sum(p);
    m_run = m_new;
    ps[lane] = p;
    __syncthreads();
    const int n = min(64, kv_end - kv0);
#pragma unroll
    for (int c = 0; c < DPL; ++c) {
      const int d = lane + c * 64;
      float a = acc[c] * alpha;
      for (int jj = 0; jj < n; ++jj)
        a = fmaf(ps[jj], v[(int64_t)(seq0 + kv0 + jj) * kv_stride + (int64_t)g * D + d], a);
      acc[c] = a;
    }
    __syncthreads();
  }
#pragma unroll
  for (int c = 0; c < DPL; ++c)
    o[((int64_t)t * Hq + h) * D + lane + c * 64] = acc[c] / l_run;
}

static hipError_t launch_attn_prefill_f32(const void* q, const void* k, const void* v,
                                          int64_t q_stride, int64_t kv_stride, void* o,
                                          const int32_t* cu, int32_t B, int64_t total_tokens,
                                          int32_t Hq, int32_t Hkv, int32_t D, float scale, bool causal,
                                          hipStream_t s) {
  const dim3 grid((unsigned)total_tokens, (unsigned)Hq);
  if (D == 128)
    hipLaunchKernelGGL((attn_prefill_f32_kernel<128>), grid, dim3(64), 0, s,
                       static_cast<const float*>(q), static_cast<const float*>(k),
                       static_cast<const float*>(v), q_stride, kv_stride, static_cast<float*>(o), cu,
                       B, Hq, Hkv, scale, (int)causal);
  else
    hipLaunchKernelGGL((attn_prefill_f32_kernel<64>), grid, dim3(64), 0, s,
                       static_cast<const float*>(q), static_cast<const float*>(k),
                       static_cast<const float*>(v), q_stride, kv_stride, static_cast<float*>(o), cu,
                       B, Hq, Hkv, scale, (int)causal);
  return hipGetLastError();
}

hipError_t launch_attn_prefill(const void* q, const void* k, const void* v, int64_t q_stride,
                               int64_t kv_stride, void* o, const int32_t* cu, int32_t B,
                               int64_t total_tokens, int32_t max_seqlen, int32_t Hq, int32_t Hkv,
                               int32_t D, float scale, bool causal, bool bf16, hipStream_t s) {
  if (!bf16)
    return launch_attn_prefill_f32(q, k, v, q_stride, kv_stride, o, cu, B, total_tokens, Hq, Hkv, D,
                                   scale, causal, s);
  const int G = Hq / Hkv;
  const int hpb = (G % 4 == 0) ? 4 : (G % 2 == 0) ? 2 : 1;
  const int BQ = 32 * (4 / hpb);
  const float sl2 = scale * kLog2e;
  // The grid launches B x ceil(max_seqlen / BQ) x HG workgroups, of which
  // only sum_b ceil(L_b / BQ) x HG have a tile; the work list launches about
  // that many (an upper bound: total_tokens / BQ + B tiles per HG) but pays a
  // small fixed cost per workgroup to find its item.  Prompts that fill less
  // than three quarters of B x max_seqlen favour the work list.
  const int64_t max_items = (total_tokens / BQ + B) * (int64_t)Hkv * (G / hpb);
  bool list = B <= kMaxListB && (double)total_tokens < 0.75 * (double)B * (double)max_seqlen;
  // OPSCALE_TUNE_PREFILL_SCHEDULE overrides the choice (0 grid, 1 list);
  // batches of more than kMaxListB prompts always use the grid.
  const int32_t force = tuning(OPSCALE_TUNE_PREFILL_SCHEDULE);
  if (force == 0) list = false;
  else if (force == 1) list = B <= kMaxListB;
  const unsigned gx = list ? (unsigned)std::min<int64_t>(0x7fffffff, max_items) : (unsigned)(B * Hkv * (G / hpb));
  const unsigned gy = list ? 1u : (unsigned)std::min<int64_t>(65535, (max_seqlen + BQ - 1) / BQ);
#define OPS_PF(DD, P)                                                                                   \
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<DD, P>), dim3(gx, gy), dim3(256), 0, s,                  \
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),                      \
                     static_cast<const __bf16*>(v), q_stride, kv_stride, static_cast<__bf16*>(o), cu, B, \
                     Hq, Hkv, hpb, sl2, (int)causal)
  if (D == 128) {
    if (list) OPS_PF(128, true);
    else OPS_PF(128, false);
  } else {
    if (list) OPS_PF(64, true);
    else OPS_PF(64, false);
  }
#undef OPS_PF
  return hipGetLastError();
}

}  // namespace opscale
