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

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBKV = 64;  // keys per K/V tile
}  // namespace

template <int D>
struct PrefillSmem {
  // K tile: 64 rows of D bf16, 16-byte chunk c of row r at chunk c ^ (r % CPR)
  // where CPR = D/8 chunks per row.  V^T tile: D rows of 64 keys (128 B), the
  // 8-byte chunk kc of row d at kc ^ (d % 16).
  static constexpr int kRowBytes = D * 2;
  static constexpr int kKBytes = kBKV * kRowBytes;
  static constexpr int kVBytes = D * kBKV * 2;
  static constexpr int kStage = kKBytes + kVBytes;
  static constexpr int kTotal = 2 * kStage;
};

template <int D>
__device__ __forceinline__ int k_swz(int r) {
  return D == 128 ? (r & 15) : ((r ^ (r >> 3)) & 7);
}

template <int D>
__global__ __launch_bounds__(256, 2) void attn_prefill_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    int64_t q_stride, int64_t kv_stride, __bf16* __restrict__ o, const int32_t* __restrict__ cu,
    int Hq, int Hkv, int hpb, float scale_log2, int causal) {
  using S = PrefillSmem<D>;
  constexpr int CPR = D / 8;          // 16-byte chunks per row
  constexpr int DSTEPS = D / 16;      // MFMA k-steps over the head dim
  constexpr int DT = D / 32;          // 32-wide output tiles over the head dim
  __shared__ __attribute__((aligned(16))) char smem_raw[S::kTotal];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;

  const int G = Hq / Hkv;
  const int nhb = G / hpb;
  const int qsub = 4 / hpb;
  const int BQ = 32 * qsub;
  const int bx = blockIdx.x;
  const int b = bx / (Hkv * nhb);
  const int g = (bx / nhb) % Hkv;
  const int hb = bx % nhb;
  const int seq0 = cu[b];
  const int L = cu[b + 1] - seq0;
  const int ntiles = (L + BQ - 1) / BQ;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = g * G + hb * hpb + wave % hpb;
  const int qs = wave / hpb;
  const int fr = lane & 31, fh = lane >> 5;

  for (int t = gridDim.y - 1 - blockIdx.y; t < ntiles; t += gridDim.y) {
    const int q_lo = t * BQ + qs * 32;          // first query of this wave
    const int q_pos = q_lo + fr;                 // this lane's query
    const int blk_q_hi = min(L, (t + 1) * BQ);   // one past the block's last query
    const int kv_end = causal ? blk_q_hi : L;
    const int nkv = (kv_end + kBKV - 1) / kBKV;

    // This wave's 32 query rows as MFMA B operand: chunk 2*s + fh of row q_pos.
    bf16x8 qf[DSTEPS];
    {
      const int rows = max(0, min(32, L - q_lo));
      const __amdgpu_buffer_rsrc_t qr = make_rsrc(
          q + (int64_t)(seq0 + q_lo) * q_stride + (int64_t)h * D,
          rows > 0 ? (uint32_t)(((int64_t)(rows - 1) * q_stride + D) * 2) : 0u);
#pragma unroll
      for (int s = 0; s < DSTEPS; ++s) {
        const u32x4 w = buffer_load16(qr, (uint32_t)(((int64_t)fr * q_stride + (2 * s + fh) * 8) * 2));
        qf[s] = __builtin_bit_cast(bf16x8, w);
      }
    }

    f32x16 acc[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) acc[i] = f32x16{};
    float m_run = -INFINITY, l_part = 0.f;

    // K tile loader (LDS DMA) and V tile loader (registers, written transposed).
    auto kv_rsrc = [&](const __bf16* base, int kv0) {
      const int rows = min(kBKV, L - kv0);
      return make_rsrc(base + (int64_t)(seq0 + kv0) * kv_stride + (int64_t)g * D,
                       (uint32_t)(((int64_t)(rows - 1) * kv_stride + D) * 2));
    };
    auto load_k = [&](int kv0, int stage) {
      const __amdgpu_buffer_rsrc_t kr = kv_rsrc(k, kv0);
      OPS_LDS char* dst = smem + stage * S::kStage;
      constexpr int ROWS_PER_LOAD = 64 / CPR;  // rows covered by one 1 KB wave load
#pragma unroll
      for (int grp = wave; grp < kBKV / ROWS_PER_LOAD; grp += 4) {
        const int r = grp * ROWS_PER_LOAD + lane / CPR;
        const int c = (lane % CPR) ^ k_swz<D>(r);
        buffer_load16_lds(kr, dst + grp * 1024, (uint32_t)(((int64_t)r * kv_stride + c * 8) * 2));
      }
    };
    // V: thread -> (key pair kp = 0..31, chunk c), 2*CPR*32/256 items per thread.
    constexpr int VITEMS = 32 * CPR / 256;  // items (key pair x chunk) per thread
    u32x4 vreg[VITEMS][2];
    auto load_v = [&](int kv0) {
      const __amdgpu_buffer_rsrc_t vr = kv_rsrc(v, kv0);
#pragma unroll
      for (int it = 0; it < VITEMS; ++it) {
        const int item = threadIdx.x + it * 256;
        const int kp = item & 31, c = item >> 5;
#pragma unroll
        for (int e = 0; e < 2; ++e)
          vreg[it][e] = buffer_load16(vr, (uint32_t)(((int64_t)(2 * kp + e) * kv_stride + c * 8) * 2));
      }
    };
    auto store_vt = [&](int stage) {
      OPS_LDS char* vt = smem + stage * S::kStage + S::kKBytes;
#pragma unroll
      for (int it = 0; it < VITEMS; ++it) {
        const int item = threadIdx.x + it * 256;
        const int kp = item & 31, c = item >> 5;
        const uint32_t a[4] = {vreg[it][0][0], vreg[it][0][1], vreg[it][0][2], vreg[it][0][3]};
        const uint32_t bb[4] = {vreg[it][1][0], vreg[it][1][1], vreg[it][1][2], vreg[it][1][3]};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = c * 8 + e;
          const uint32_t lo = (e & 1) ? (a[e >> 1] >> 16) : (a[e >> 1] & 0xffffu);
          const uint32_t hi = (e & 1) ? (bb[e >> 1] & 0xffff0000u) : (bb[e >> 1] << 16);
          const int kc = (2 * kp) >> 2;  // 8-byte chunk of 4 keys
          const int off = d * (kBKV * 2) + ((kc ^ (d & 15)) << 3) + ((2 * kp) & 3) * 2;
          *reinterpret_cast<OPS_LDS uint32_t*>(vt + off) = lo | hi;
        }
      }
    };

    if (nkv > 0) {
      load_k(0, 0);
      load_v(0);
      store_vt(0);
    }
    for (int it = 0; it < nkv; ++it) {
      const int kv0 = it * kBKV;
      wait_vmem();
      __syncthreads();
      const bool more = it + 1 < nkv;
      if (more) {
        load_k(kv0 + kBKV, (it + 1) & 1);
        load_v(kv0 + kBKV);
      }
      const OPS_LDS char* ks = smem + (it & 1) * S::kStage;
      const OPS_LDS char* vts = ks + S::kKBytes;
      // Skip tiles that are entirely in this wave's causal future.
      const bool active = !(causal && kv0 > q_lo + 31) && q_lo < L;
      if (active) {
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
        // scale into the log2 domain and mask
        const bool need_mask = (causal && kv0 + kBKV - 1 > q_lo) || (kv0 + kBKV > L);
        float tmax = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            float sv = st[kb][e] * scale_log2;
            if (need_mask) {
              const int key = kv0 + kb * 32 + (e >> 2) * 8 + fh * 4 + (e & 3);
              if (key >= L || (causal && key > q_pos)) sv = -INFINITY;
            }
            st[kb][e] = sv;
            tmax = fmaxf(tmax, sv);
          }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float m_new = fmaxf(m_run, tmax);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = fast_exp2(m_run - m_use);
        m_run = m_new;
        float psum = 0.f;
        bf16x8 pf[4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float p = fast_exp2(st[kb][e] - m_use);
            psum += p;
            pf[kb * 2 + (e >> 3)][e & 7] = (__bf16)p;
          }
        l_part = l_part * alpha + psum;
#pragma unroll
        for (int i = 0; i < DT; ++i) acc[i] *= alpha;
        // the next V tile goes to the other stage now, before the PV product,
        // so its registers are free again for the accumulators
        if (more) store_vt((it + 1) & 1);
        // O^T[d][i] += sum_key V^T[d][key] P^T[key][i]
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const int d = dt * 32 + fr;
          const OPS_LDS char* row = vts + d * (kBKV * 2);
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            const int kc0 = 4 * s + fh, kc1 = 4 * s + 2 + fh;
            const u32x2 lo = *reinterpret_cast<const OPS_LDS u32x2*>(row + ((kc0 ^ (d & 15)) << 3));
            const u32x2 hi = *reinterpret_cast<const OPS_LDS u32x2*>(row + ((kc1 ^ (d & 15)) << 3));
            const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
            acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), pf[s],
                                                             acc[dt], 0, 0, 0);
          }
        }
      } else if (more) {
        store_vt((it + 1) & 1);
      }
    }

    // normalize and store: lane owns query q_pos; acc[dt][e] is
    // d = dt*32 + (e/4)*8 + fh*4 + e%4.
    const float l_tot = l_part + __shfl_xor(l_part, 32, 64);
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
    __syncthreads();  // the next tile reuses the LDS stages
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
  const unsigned gx = (unsigned)(B * Hkv * (G / hpb));
  const unsigned gy = (unsigned)std::min<int64_t>(65535, (max_seqlen + BQ - 1) / BQ);
  const float sl2 = scale * kLog2e;
  if (D == 128)
    hipLaunchKernelGGL((attn_prefill_bf16_kernel<128>), dim3(gx, gy), dim3(256), 0, s,
                       static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                       static_cast<const __bf16*>(v), q_stride, kv_stride, static_cast<__bf16*>(o),
                       cu, Hq, Hkv, hpb, sl2, (int)causal);
  else
    hipLaunchKernelGGL((attn_prefill_bf16_kernel<64>), dim3(gx, gy), dim3(256), 0, s,
                       static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                       static_cast<const __bf16*>(v), q_stride, kv_stride, static_cast<__bf16*>(o),
                       cu, Hq, Hkv, hpb, sl2, (int)causal);
  return hipGetLastError();
}

}  // namespace opscale
