// Linear layers y[M,N] = x[M,K] W[N,K]^T (+ bias): QKV, O, gate-up and down
// projections of the decoder layer.
//
// bf16 path: MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation.  A 256x256
// block tile is staged through an LDS ring in BK-wide K slices; the next slices
// are fetched with buffer_load ... lds (HBM/L2 -> LDS without passing through
// registers) while the current one feeds the matrix cores.  Large problems
// use four waves of 128x128 sub-tiles, one per SIMD, with the accumulators in
// AGPRs (gemm_bf16_w4_kernel); the eight-wave form of the same tile (two waves
// of 128x64 per SIMD) serves the grouped mixture-of-experts GEMMs.  Problems
// whose last round of 256x256 tiles would be mostly idle take 192x256 or
// 256x128 tiles; decode-sized M splits K.  Rows
// and K columns beyond the matrix read as zeros through the buffer
// descriptor's range check, so ragged M, N and K need no separate code path.
//
// Both operands are K-contiguous, which is what an MFMA operand lane wants: a
// lane holds 8 consecutive k of one row.  The W tile is the MFMA "A" operand
// and the x tile the "B" operand, so each accumulator lane owns one output row
// m and runs of 4 consecutive columns n, stored as 8-byte chunks.
//
// fp32 path: a plain LDS-tiled FMA kernel (exact fp32 products and sums).
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace opscale {

namespace {

constexpr int kNumCUs = 256;  // MI355X compute units
constexpr int64_t kGroupBytes = (int64_t)16 << 20;  // x rows per tile group (see tile_group_rows)
constexpr int64_t kSplitKMaxM = 2048;  // split-K is for small M (decode batches)

// Tile configuration: BM x BN block tile, K in slices of BK, WGM x WGN waves
// (each owns a (BM/WGM) x (BN/WGN) sub-tile), STAGES-deep LDS ring.
// DEEP: the ring keeps STAGES - 1 slices in flight while a slice is used
// (decode-sized M, where the loop waits on memory, not on the matrix cores);
// otherwise the next slice is made visible one step early so its first
// fragment reads overlap the current slice's last MFMAs.
template <int BM_, int BN_, int BK_, int WGM_, int WGN_, int STAGES_, bool DEEP_ = false>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WGM = WGM_, WGN = WGN_, STAGES = STAGES_;
  static constexpr bool DEEP = DEEP_;
  static constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile (m x n)
  static constexpr int kThreads = WGM * WGN * 64;
  static constexpr int kWaves = WGM * WGN;
  static constexpr int kRowBytes = BK * 2;              // one LDS row = BK bf16
  static constexpr int kCPR = BK / 8;                   // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 64 / kCPR;        // rows one 1 KB wave load covers
  static constexpr int kStageBytes = (BM + BN) * kRowBytes;
  static constexpr int kLdsBytes = STAGES * kStageBytes;
  static constexpr int kLoadsPerTile = (BM + BN) / kRowsPerLoad / kWaves;  // per wave
  static_assert(BM % (kRowsPerLoad * kWaves) == 0 && BN % (kRowsPerLoad * kWaves) == 0,
                "each operand's rows must split evenly over the waves");
  // The fragment double buffer alternates by k-step within a slice and
  // restarts at buffer 0 in the next, so a slice must hold an even number of
  // 32-wide k-steps; the LDS swizzle assumes 128-byte rows.
  static_assert(BK == 64, "64-wide K slices: two 32-wide k-steps of 128-byte rows");
  static_assert(kLoadsPerTile * (STAGES - 2 > 0 ? STAGES - 2 : 0) <= 63, "vmcnt range");
};

using CfgBig8 = GemmCfg<256, 256, 64, 2, 4, 2>;    // 8 waves of 128x64, 2 x 64 KB stages
using CfgT192 = GemmCfg<192, 256, 64, 2, 4, 2>;    // 8 waves of 96x64, 2 x 56 KB stages
using CfgMid = GemmCfg<256, 128, 64, 2, 2, 3>;     // 4 waves of 128x64, 3 x 48 KB stages
using CfgW4 = GemmCfg<256, 256, 64, 2, 2, 2>;      // 4 waves of 128x128, 2 x 64 KB stages
using CfgRow64 = GemmCfg<64, 256, 64, 1, 4, 2>;    // 4 waves of 64x64, 2 x 40 KB stages (few rows)
// split-K tiles for decode-sized M: a K range is short, so the ring is deep
using CfgSk64 = GemmCfg<64, 256, 64, 1, 4, 4, true>;    // M <= 64: 4 waves of 64x64, 4 x 40 KB stages
using CfgSk128 = GemmCfg<128, 256, 64, 2, 4, 3, true>;  // M <= 256: 8 waves of 64x64, 3 x 48 KB stages


// 16-byte chunk c of LDS row r is stored at physical chunk c ^ swz(r).
// gfx950 LDS has 64 banks of 4 bytes and serves a 16-byte-per-lane read in
// four passes of 16 lanes: pass 2 * (lane / 32) + parity of bits 2..4 of the
// lane (lanes in 4-lane blocks, blocks of odd and even bit parity alternating;
// measured).  A 16x16x32 operand read puts row lane % 16 and logical chunk
// 4 ks + lane / 16 in each lane, so a pass holds 8 rows of one parity class at
// each of two chunks; XOR with the row mod 8 gives those 16 lanes 16
// distinct 16-byte bank groups for both k-steps of a 64-wide slice.  swz depends only
// on the row mod 16, i.e. on the lane, so one per-lane offset per K step
// serves every 16-row fragment of a wave (the rest is an immediate offset).
template <int CPR>
__device__ __forceinline__ int swz(int r) {
  static_assert(CPR == 8, "128-byte rows");
  return r & 7;
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt in bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// One BK-wide slice of ROWS rows of a K-contiguous bf16 matrix (descriptor
// based at the tile's first row) into an LDS stage region.  Wave w issues
// loads w, w + waves, ...; lane p of a load writes LDS bytes [p*16, p*16+16)
// of its 1 KB group: row p / CPR, physical chunk p % CPR.
// A row that must read as zeros (past the end of a grouped operand).
constexpr uint32_t kNoRow = 0xffffffffu;

// row_off[g]: byte offset of the row this lane loads in its g-th load group
// (kNoRow: a row that reads as zeros).
template <class C, int ROWS>
__device__ __forceinline__ void load_slice(__amdgpu_buffer_rsrc_t rsrc, OPS_LDS char* lds, const uint32_t* row_off,
                                           int K, int k0, int wave, int lane) {
  const int rl = lane / C::kCPR, pc = lane % C::kCPR;
  constexpr int kPerWave = ROWS / C::kRowsPerLoad / C::kWaves;
#pragma unroll
  for (int g = 0; g < kPerWave; ++g) {
    const int grp = g * C::kWaves + wave;
    const int r = grp * C::kRowsPerLoad + rl;
    const int c = pc ^ swz<C::kCPR>(r);
    const int k = k0 + c * 8;
    const uint32_t voff = (k < K && row_off[g] != kNoRow) ? row_off[g] + (uint32_t)k * 2u : kOobOffset;
    buffer_load16_lds<kNoL1>(rsrc, lds + grp * 1024, voff);
  }
}

template <class C>
__device__ __forceinline__ bf16x8 lds_frag(const OPS_LDS char* p) {
  return *reinterpret_cast<const OPS_LDS bf16x8*>(p);
}

}  // namespace

// Tile (tm, tn) of plain-GEMM tile id tid in grouped order: group_m
// tile-rows sweep the tile-columns together, so a W column-block is fetched
// once per group and reused from L2 / MALL by every tile-row of the group
// while the group's x rows stay cache resident.
__device__ __forceinline__ void tile_coords(uint32_t tid, int tiles_m, int tiles_n, int group_m, int& tm, int& tn) {
  const int group = tid / (group_m * tiles_n);
  const int first_m = group * group_m;
  const int gsize = min(tiles_m - first_m, group_m);
  const int in_group = tid % (group_m * tiles_n);
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// Split-K (splits > 1): workgroup blockIdx.x / tiles takes the K range
// [split * kchunk, (split + 1) * kchunk) and writes its fp32 partial tile to
// part[split][M][N] (no bias); a second kernel sums the splits in order.
//
// Split tail (tail_cnt > 0): workgroups [0, dp_cnt) take whole tiles 0 ..
// dp_cnt - 1 (full K, results to y); the rest take the K ranges of the last
// tail_cnt tiles: item b (from dp_cnt) covers tile dp_cnt + b % tail_cnt, K
// range b / tail_cnt, and writes its fp32 tile compactly to
// part[(split * tail_cnt + tile - dp_cnt) * BM * BN] (row-major BM x BN); a
// second kernel sums those in split order.  Runs a launch whose last round
// would be mostly idle at a fraction of a tile's time.
//
// GROUPED (one GEMM per expert of a mixture-of-experts layer): the output
// rows are grouped by expert, expert e owning rows [rows[e], rows[e + 1]) in
// tiles tiles[e] .. tiles[e + 1] - 1 of BM rows; workgroup (tile t, column
// block n) multiplies by W + e * w_stride, and output row m reads x row
// gather[m] (m itself when gather is null).  x then has x_rows rows.
struct GroupedGemm {
  const int32_t* gather;  // output row -> x row (null: the identity)
  const int32_t* rows;    // [E + 1]
  const int32_t* tiles;   // [E + 1]
  int E;
  int x_rows;
  int64_t w_stride;       // elements from one expert's W to the next
  // > 0: W is a gate-up projection [2F, K] (gate rows first) and y the SwiGLU
  // activation [rows, F]: output column c of the GEMM is gate row c / 2 (even
  // c) or up row F + c / 2 (odd c), so each lane's runs of 4 columns hold two
  // (gate, up) pairs and the epilogue stores silu(gate) * up.  N = 2F.
  int swiglu_f;
};

template <class C, bool GROUPED = false>
__global__ __launch_bounds__(C::kThreads, 1) void gemm_bf16_kernel(const __bf16* __restrict__ x,
                                                                   const __bf16* __restrict__ W,
                                                                   const __bf16* __restrict__ bias,
                                                                   __bf16* __restrict__ y, int M, int N,
                                                                   int K_total, int group_m, int kchunk,
                                                                   float* __restrict__ part, GroupedGemm gg,
                                                                   int dp_cnt, int tail_cnt) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, WM = C::WM, WN = C::WN, S = C::STAGES;
  // 16x16x32 MFMAs: half the length of a 32x32x16 one for the same work per
  // k-window, so the next fragments' LDS reads and the loads find twice the
  // issue slots between them (measured 0-2 % faster on every shape here)
  constexpr int MI = 16;
  constexpr int TM = WM / MI, TN = WN / MI;  // MFMA tiles per wave

  const int tiles_n = (N + BN - 1) / BN;
  const int ld = K_total;
  int m0, n0, m_rows, split = 0;
  int kc = kchunk;                  // K elements per split
  float* tile_part = nullptr;       // split tail: this item's compact partial tile
  if constexpr (GROUPED) {
    // Work items in order expert, column block, tile-row of the expert, so
    // an expert's tile-rows use one W column block back to back; spread over
    // the XCDs in contiguous ranges of the items that exist (the grid is an
    // upper bound; the workgroups past it return).
    const int total = gg.tiles[gg.E] * tiles_n;
    if ((int)blockIdx.x >= total) return;
    const int id = (int)xcd_remap(blockIdx.x, (uint32_t)total);
    int lo = 0, hi = gg.E;  // gg.tiles[lo] * tiles_n <= id < gg.tiles[hi] * tiles_n
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (gg.tiles[mid] * tiles_n <= id) lo = mid;
      else hi = mid;
    }
    const int tr_e = gg.tiles[lo + 1] - gg.tiles[lo];  // tile-rows of expert lo (>= 1)
    const int local = id - gg.tiles[lo] * tiles_n;
    const int tn = local / tr_e, tr = local - tn * tr_e;
    n0 = tn * BN;
    m0 = gg.rows[lo] + tr * BM;
    m_rows = min(BM, gg.rows[lo + 1] - m0);
    W += lo * gg.w_stride;
  } else {
    const int tiles_m = (M + BM - 1) / BM;
    const int tiles = tiles_m * tiles_n;
    uint32_t tid;
    if (tail_cnt == 0) {
      split = blockIdx.x / tiles;
      tid = xcd_remap(blockIdx.x - split * tiles, (uint32_t)tiles);
    } else if ((int)blockIdx.x < dp_cnt) {
      tid = xcd_remap(blockIdx.x, (uint32_t)dp_cnt);
      kc = K_total;
    } else {
      const int b = blockIdx.x - dp_cnt;
      split = b / tail_cnt;
      const int t = (int)xcd_remap(b - split * tail_cnt, (uint32_t)tail_cnt);
      tid = dp_cnt + t;
      tile_part = part + ((int64_t)split * tail_cnt + t) * BM * BN;
    }
    int tm, tn;
    tile_coords(tid, tiles_m, tiles_n, group_m, tm, tn);
    m0 = tm * BM;
    n0 = tn * BN;
    m_rows = min(BM, M - m0);
  }
  // this workgroup's K range: K elements starting at k_begin, rows ld apart
  const int k_begin = split * kc;
  const int K = min(K_total - k_begin, kc);

  // wave index as a scalar: the LDS destinations of the loads are then
  // wave-uniform without a readfirstlane per load
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int wm = wave % C::WGM, wn = wave / C::WGM;

  // x: the tile's rows (grouped: the gathered rows of the whole operand)
  const __amdgpu_buffer_rsrc_t xr =
      GROUPED ? make_rsrc(x + k_begin, (uint32_t)(((int64_t)gg.x_rows - 1) * ld * 2 + (int64_t)K * 2))
              : make_rsrc(x + (int64_t)m0 * ld + k_begin, (uint32_t)(((int64_t)(m_rows - 1) * ld + K) * 2));
  // W: the tile's rows (fused SwiGLU: the expert's whole gate-up weight)
  const bool fused = GROUPED && gg.swiglu_f > 0;
  const __amdgpu_buffer_rsrc_t wr =
      fused ? make_rsrc(W + k_begin, (uint32_t)(((int64_t)N - 1) * ld * 2 + (int64_t)K * 2))
            : make_rsrc(W + (int64_t)n0 * ld + k_begin, (uint32_t)(((int64_t)(min(BN, N - n0) - 1) * ld + K) * 2));
  // byte offsets of the rows this lane loads (per load group)
  constexpr int LX = BM / C::kRowsPerLoad / C::kWaves, LW = BN / C::kRowsPerLoad / C::kWaves;
  uint32_t xro[LX], wro[LW];
#pragma unroll
  for (int g = 0; g < LX; ++g) {
    const int r = (g * C::kWaves + wave) * C::kRowsPerLoad + lane / C::kCPR;
    if constexpr (GROUPED) {
      const int src = r < m_rows ? (gg.gather ? gg.gather[m0 + r] : m0 + r) : -1;
      xro[g] = src >= 0 ? (uint32_t)((int64_t)src * ld * 2) : kNoRow;
    } else {
      xro[g] = (uint32_t)((int64_t)r * ld * 2);
    }
  }
#pragma unroll
  for (int g = 0; g < LW; ++g) {
    const int r = (g * C::kWaves + wave) * C::kRowsPerLoad + lane / C::kCPR;
    if (fused) {
      const int c = n0 + r;  // interleaved column: gate row c / 2, up row F + c / 2
      wro[g] = c < N ? (uint32_t)((int64_t)((c & 1) ? gg.swiglu_f + (c >> 1) : (c >> 1)) * ld * 2) : kNoRow;
    } else {
      wro[g] = (uint32_t)((int64_t)r * ld * 2);
    }
  }

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{};

  const int nk = (K + BK - 1) / BK;
  auto stage_x = [&](int s) { return smem + s * C::kStageBytes; };
  auto stage_w = [&](int s) { return smem + s * C::kStageBytes + BM * C::kRowBytes; };
  auto load = [&](int kt) {
    load_slice<C, BM>(xr, stage_x(kt % S), xro, K, kt * BK, wave, lane);
    load_slice<C, BN>(wr, stage_w(kt % S), wro, K, kt * BK, wave, lane);
  };

#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < nk) load(s);

  // operand lane roles: row fr of a 16-row fragment, 8-k chunk fh of 32
  const int fr = lane & (MI - 1), fh = lane / MI;
  constexpr int KS = BK / 32;  // MFMA k-steps per slice
  // per-lane byte offset of this lane's 16-byte fragment row in k-step ks
  int lane_off[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) lane_off[ks] = fr * C::kRowBytes + (((4 * ks + fh) ^ swz<C::kCPR>(fr)) << 4);
  // the x slice sits first in a stage, the W slice after it
  const int x_row0 = wm * WM * C::kRowBytes, w_row0 = BM * C::kRowBytes + wn * WN * C::kRowBytes;

  bf16x8 a[2][TN], b[2][TM];
  auto frags = [&](const OPS_LDS char* st, int ks, int buf) {
#pragma unroll
    for (int i = 0; i < TN; ++i) a[buf][i] = lds_frag<C>(st + w_row0 + i * MI * C::kRowBytes + lane_off[ks]);
#pragma unroll
    for (int j = 0; j < TM; ++j) b[buf][j] = lds_frag<C>(st + x_row0 + j * MI * C::kRowBytes + lane_off[ks]);
  };
  // The MFMAs of the last k-step of slice kt with the loads of slice kt + 2
  // interleaved, one load after each MFMA, so no wave issues its loads in one
  // burst (the issue of a stalled load would hold back the MFMAs behind it).
  // Past the last slice the loads are out of range (they read zeros) and go
  // to the stage no wave reads any more.
  auto mfmas_loading = [&](int buf, int kt) {
    constexpr int MF = TN * TM, L = C::kLoadsPerTile;
    OPS_LDS char* dst = smem + ((kt + 1 < nk ? kt : kt + 1) & 1) * C::kStageBytes;
    const int rl = lane / C::kCPR, pc = lane % C::kCPR;
    const int k0 = (kt + 2) * BK;
    const bool more = kt + 2 < nk;
#pragma unroll
    for (int q = 0; q < (MF > L ? MF : L); ++q) {
      if (q < MF) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[buf][i], b[buf][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      if (q < L) {
        const bool isx = q < LX;
        const int grp = (isx ? q : q - LX) * C::kWaves + wave;
        const int r = grp * C::kRowsPerLoad + rl;
        const int k = k0 + ((pc ^ swz<C::kCPR>(r)) << 3);
        const uint32_t ro = isx ? xro[q < LX ? q : 0] : wro[q >= LX ? q - LX : 0];
        const uint32_t voff = (more && k < K && ro != kNoRow) ? ro + (uint32_t)k * 2u : kOobOffset;
        buffer_load16_lds<kNoL1>(isx ? xr : wr, dst + (isx ? 0 : BM * C::kRowBytes) + grp * 1024, voff);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
  };
  // The next k-step's fragment reads (issued just before, in the same block)
  // go one after each MFMA: left to itself the scheduler puts them after the
  // MFMAs, and the next k-step then waits for a whole LDS round trip.
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[buf][i], b[buf][j], acc[i][j], 0, 0, 0);
#pragma unroll
    for (int q = 0; q < TN * TM; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (q < TN + TM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
  };

  // vmcnt <= n loads of this wave (n a multiple of kLoadsPerTile, < S slices)
  auto wait_slices = [&](int n) {
    constexpr int L = C::kLoadsPerTile;
    if (n <= 0) wait_vmcnt<0>();
    else if (n == 1) wait_vmcnt<L>();
    else if (n == 2) wait_vmcnt<(S > 2 ? 2 : 1) * L>();
    else wait_vmcnt<(S > 3 ? 3 : 1) * L>();
  };
  if constexpr (C::DEEP) {
    static_assert(S >= 3 && S <= 4, "deep ring of 3 or 4 stages");
    // Slices kt + 1 .. kt + S - 1 are in flight while slice kt is used; the
    // stage of slice kt - 1 is refilled right after the barrier that ends it.
    wait_slices(min(S - 2, nk - 1));
    barrier_keep_loads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + S - 1 < nk) load(kt + S - 1);
      const OPS_LDS char* st = smem + (kt % S) * C::kStageBytes;
      frags(st, 0, 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) frags(st, ks + 1, (ks + 1) & 1);
        mfmas(ks & 1);
      }
      // slice kt + 1 landed: the loads issued after it stay in flight
      if (kt + 1 < nk) wait_slices(min(S - 2, nk - 2 - kt));
      barrier_keep_loads();
    }
  } else if constexpr (S == 2) {
    // Slice kt + 1 is made visible before the last k-step of slice kt: that
    // step already reads slice kt + 1's first fragments, and the MFMAs issued
    // just before the barrier keep the matrix cores busy while the waves
    // meet.  Slice kt + 2 is then loaded into the stage slice kt used (every
    // wave has read its last fragments of it before the barrier).
    wait_vmcnt<0>();
    __syncthreads();
    if (nk > 1) load(1);
    frags(smem, 0, 0);
    for (int kt = 0; kt < nk; ++kt) {
      const OPS_LDS char* st = smem + (kt & 1) * C::kStageBytes;
      const OPS_LDS char* st_next = smem + ((kt + 1) & 1) * C::kStageBytes;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int nb = (ks + 1) & 1;
        if (ks + 1 < KS) {
          frags(st, ks + 1, nb);
        } else if (kt + 1 < nk) {
          wait_vmcnt<0>();
          __syncthreads();
          frags(st_next, 0, nb);
        }
        if (ks == KS - 1) mfmas_loading(ks & 1, kt);
        else mfmas(ks & 1);
      }
    }
  } else {
    // Look-ahead pipeline: at the top of iteration kt slice kt + 1 is made
    // visible, so the last k-step of slice kt already reads slice kt + 1's
    // first fragments and the matrix cores never wait on the barrier.
    if (S > 2 && nk > S - 2) wait_vmcnt<C::kLoadsPerTile * (S > 2 ? S - 2 : 0)>();
    else wait_vmcnt<0>();
    __syncthreads();
    frags(smem, 0, 0);
    for (int kt = 0; kt < nk; ++kt) {
      if (S > 3 && kt + S - 2 < nk) wait_vmcnt<C::kLoadsPerTile * (S > 3 ? S - 3 : 0)>();
      else wait_vmcnt<0>();
      __syncthreads();
      if (kt + S - 1 < nk) load(kt + S - 1);
      const OPS_LDS char* st = smem + (kt % S) * C::kStageBytes;
      const OPS_LDS char* st_next = smem + ((kt + 1) % S) * C::kStageBytes;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int nb = (ks + 1) & 1;
        if (ks + 1 < KS) frags(st, ks + 1, nb);
        else if (kt + 1 < nk) frags(st_next, 0, nb);
        mfmas(ks & 1);
      }
    }
  }

  wait_vmem();  // no LDS DMA may still be in flight when the workgroup ends

  // Epilogue.  acc[i][j] element e: n = n0 + wn*WN + i*16 + fh*4 + e,
  // m = m0 + wm*WM + j*16 + fr.  Four consecutive n per lane -> one 8-byte store
  // (one 16-byte store of fp32 partials under split-K).
  if (tile_part) {
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int r = wm * WM + j * MI + fr;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int c = wn * WN + i * MI + fh * 4;
        *reinterpret_cast<f32x4*>(tile_part + r * BN + c) = acc[i][j];
      }
    }
    return;
  }
  if (part && tail_cnt == 0) {
    float* pbase = part + (int64_t)split * M * N;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int m = m0 + wm * WM + j * MI + fr;
      if (m - m0 >= m_rows) continue;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int n = n0 + wn * WN + i * MI + fh * 4;
        if (n >= N) continue;
        *reinterpret_cast<f32x4*>(pbase + (int64_t)m * N + n) = acc[i][j];
      }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm * WM + j * MI + fr;
    if (m - m0 >= m_rows) continue;
    if (fused) {
      // two (gate, up) pairs per lane: act[m][n / 2], act[m][n / 2 + 1]
      __bf16* arow = y + (int64_t)m * gg.swiglu_f;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int n = n0 + wn * WN + i * MI + fh * 4;
        if (n >= N) continue;
        const float g0 = acc[i][j][0], u0 = acc[i][j][1], g1 = acc[i][j][2], u1 = acc[i][j][3];
        const float a0 = g0 / (1.f + __expf(-g0)) * u0, a1 = g1 / (1.f + __expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(arow + (n >> 1)) = pack_bf2(a0, a1);
      }
      continue;
    }
    __bf16* yrow = y + (int64_t)m * N;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      {
        const int n = n0 + wn * WN + i * MI + fh * 4;
        if (n >= N) continue;
        float v0 = acc[i][j][0], v1 = acc[i][j][1];
        float v2 = acc[i][j][2], v3 = acc[i][j][3];
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

// One MFMA 16x16x32 on an accumulator held in AGPRs.  Issued from inline
// assembly so that the 64 accumulators of a 128x128 wave tile stay in place:
// with the builtin the register allocator rotated them through AGPR copies and
// spilled.  An assembly statement with side effects also fixes the order of
// the memory instructions around it, which places the fragment reads and the
// tile loads between the MFMAs exactly as written.
__device__ __forceinline__ void mfma_agpr(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// An accumulator's four values into VGPRs.  Read through assembly as well:
// were the epilogue's arithmetic to read the AGPRs directly, the compiler
// would give the accumulators VGPR homes and copy them around every MFMA.
__device__ __forceinline__ f32x4 agpr_read(const f32x4& acc) {
  f32x4 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(acc[e]));
  return v;
}

// The 256x256 tile as four waves of 128x128, one wave per SIMD.  With two
// waves per SIMD (gemm_bf16_kernel's eight-wave form) the older wave takes
// the matrix core first and then waits at the slice barrier while the younger
// one finishes alone; here every SIMD runs one wave and the slice's fragment
// reads fall from 192 to 128 KB per workgroup.  Swizzle, loads, split tail
// and epilogue are those of gemm_bf16_kernel.  A k-step is 64 MFMAs; the 16
// fragment reads of the next k-step go one after each of its first 16 MFMAs
// (in the order the next k-step consumes them), and in the last k-step of a
// slice 16 loads go one after every fourth MFMA.
//
// The LDS ring is five 32 KB half-slices (160 KB) rather than two 64 KB
// slices: the x half and the W half of a slice rotate through the buffers
// separately, so once slice kt is read its buffers take the W half of slice
// kt + 2 and the x half of slice kt + 3.  About 1.5 slices (96 KB) are in
// flight per CU instead of at most one, and the x halves get two slices of
// time to land.  The loads are latency bound: the tile-load pattern alone
// moves 18 TB/s over the chip this way against 13.7 TB/s with two stages.
template <class C, bool XLEAD>
__global__ __launch_bounds__(C::kThreads, 1) void gemm_bf16_w4_kernel(const __bf16* __restrict__ x,
                                                                      const __bf16* __restrict__ W,
                                                                      const __bf16* __restrict__ bias,
                                                                      __bf16* __restrict__ y, int M, int N,
                                                                      int K_total, int group_m, int kchunk,
                                                                      float* __restrict__ part, GroupedGemm,
                                                                      int dp_cnt, int tail_cnt) {
  static_assert(C::kWaves == 4 && C::WM == 128 && C::WN == 128 && !C::DEEP, "four waves of 128x128");
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  OPS_LDS char* smem = (OPS_LDS char*)smem_raw;
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, WM = C::WM, WN = C::WN;
  constexpr int MI = 16, TM = WM / MI, TN = WN / MI, KS = BK / 32;

  const int tiles_n = (N + BN - 1) / BN;
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles = tiles_m * tiles_n;
  const int ld = K_total;
  int split = 0, kc = kchunk;
  float* tile_part = nullptr;
  uint32_t tid;
  if (tail_cnt == 0) {
    split = blockIdx.x / tiles;
    tid = xcd_remap(blockIdx.x - split * tiles, (uint32_t)tiles);
  } else if ((int)blockIdx.x < dp_cnt) {
    tid = xcd_remap(blockIdx.x, (uint32_t)dp_cnt);
    kc = K_total;
  } else {
    const int b = blockIdx.x - dp_cnt;
    split = b / tail_cnt;
    const int t = (int)xcd_remap(b - split * tail_cnt, (uint32_t)tail_cnt);
    tid = dp_cnt + t;
    tile_part = part + ((int64_t)split * tail_cnt + t) * BM * BN;
  }
  int tm, tn;
  tile_coords(tid, tiles_m, tiles_n, group_m, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int m_rows = min(BM, M - m0);
  const int k_begin = split * kc;
  const int K = min(K_total - k_begin, kc);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int wm = wave % C::WGM, wn = wave / C::WGM;
  const __amdgpu_buffer_rsrc_t xr =
      make_rsrc(x + (int64_t)m0 * ld + k_begin, (uint32_t)(((int64_t)(m_rows - 1) * ld + K) * 2));
  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc(W + (int64_t)n0 * ld + k_begin, (uint32_t)(((int64_t)(min(BN, N - n0) - 1) * ld + K) * 2));
  constexpr int LX = BM / C::kRowsPerLoad / C::kWaves, LW = BN / C::kRowsPerLoad / C::kWaves;
  constexpr int L = LX + LW;
  static_assert(L * 4 == TM * TN, "one load after every fourth MFMA of a k-step");
  uint32_t xro[LX], wro[LW];
#pragma unroll
  for (int g = 0; g < LX; ++g) xro[g] = (uint32_t)(((g * C::kWaves + wave) * C::kRowsPerLoad + lane / C::kCPR) * ld * 2);
#pragma unroll
  for (int g = 0; g < LW; ++g) wro[g] = (uint32_t)(((g * C::kWaves + wave) * C::kRowsPerLoad + lane / C::kCPR) * ld * 2);

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{};

  const int nk = (K + BK - 1) / BK;
  // The ring holds five half-slices of HB bytes: the lead operand's rows of
  // slice s (x if XLEAD, else W) are half 2s, the other operand's half 2s + 1,
  // and half u lives in buffer u mod 5.
  constexpr int HB = BM * C::kRowBytes;
  // load g (0 .. 7) of the x (ISX) or W half of slice s into buffer dst
  // (zeros past the end)
  auto load_half = [&](auto isx_c, OPS_LDS char* dst, int s, int g) {
    constexpr bool ISX = decltype(isx_c)::value;
    const int rl = lane / C::kCPR, pc = lane % C::kCPR;
    const int grp = g * C::kWaves + wave;
    const int r = grp * C::kRowsPerLoad + rl;
    // (a slice past the end starts at K, so every lane's k is out of range:
    // one select per load and no branch)
    const int k = (s < nk ? s * BK : K) + ((pc ^ swz<C::kCPR>(r)) << 3);
    const uint32_t voff = k < K ? (ISX ? xro[g] : wro[g]) + (uint32_t)k * 2u : kOobOffset;
    buffer_load16_lds<kNoL1>(ISX ? xr : wr, dst + grp * 1024, voff);
  };
  using TL = std::integral_constant<bool, XLEAD>;   // the lead operand (true: x)
  using TF = std::integral_constant<bool, !XLEAD>;  // the other one
  const int fr = lane & (MI - 1), fh = lane / MI;
  int lane_off[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) lane_off[ks] = fr * C::kRowBytes + (((4 * ks + fh) ^ swz<C::kCPR>(fr)) << 4);
  const int x_row0 = wm * WM * C::kRowBytes, w_row0 = wn * WN * C::kRowBytes;

  bf16x8 a[2][TN], b[2][TM];
  // fragment read r (0 .. TN + TM - 1) of a k-step from the x half rx and the
  // W half rw, in the order the MFMAs (i outer, j inner) first need them:
  // b0, a0, b1 .. b7, a1 .. a7
  auto read_frag = [&](const OPS_LDS char* rx, const OPS_LDS char* rw, int ks, int buf, int r) {
    if (r == 0) b[buf][0] = lds_frag<C>(rx + x_row0 + lane_off[ks]);
    else if (r == 1) a[buf][0] = lds_frag<C>(rw + w_row0 + lane_off[ks]);
    else if (r < TM + 1) b[buf][r - 1] = lds_frag<C>(rx + x_row0 + (r - 1) * MI * C::kRowBytes + lane_off[ks]);
    else a[buf][r - TM] = lds_frag<C>(rw + w_row0 + (r - TM) * MI * C::kRowBytes + lane_off[ks]);
  };
  // one k-step on fragment buffer buf; READ: the next k-step's fragments
  // (halves rx / rw, k-step rks) into buf ^ 1; LOAD: the other operand's half
  // of slice kt + 2 into df, then the lead operand's half of slice kt + 3
  // into dl (in this order: the next barrier waits for the first and leaves
  // the second in flight)
  auto kstep = [&](auto buf_c, auto read_c, auto load_c, const OPS_LDS char* rx, const OPS_LDS char* rw, int rks,
                   OPS_LDS char* df, OPS_LDS char* dl, int kt) {
    constexpr int buf = decltype(buf_c)::value;
    constexpr bool READ = decltype(read_c)::value, LOAD = decltype(load_c)::value;
    // This k-step's fragments were read one k-step ago and have landed; with
    // the counter cleared the compiler needs no wait inside the MFMA run (it
    // could not name one that lets the new reads stay in flight: the LDS
    // counter holds at most 15).
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
#pragma unroll
    for (int q = 0; q < TN * TM; ++q) {
      mfma_agpr(acc[q / TM][q % TM], a[buf][q / TM], b[buf][q % TM]);
      if (READ && q < TN + TM) read_frag(rx, rw, rks, buf ^ 1, q);
      if (LOAD && (q & 3) == 3) {
        const int l = q >> 2;
        if (l < LW) load_half(TF{}, df, kt + 2, l);
        else load_half(TL{}, dl, kt + 3, l - LW);
      }
    }
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using T = std::true_type;
  using F = std::false_type;
  static_assert(KS == 2, "two k-steps per slice");
  static_assert(BM == BN && LX == 8 && LW == 8, "square tile: x and W halves of 8 loads per wave");

  // prologue: halves 0 .. 4 (slices 0 and 1, the lead half of slice 2)
#pragma unroll
  for (int g = 0; g < LX; ++g) load_half(TL{}, smem, 0, g);
#pragma unroll
  for (int g = 0; g < LW; ++g) load_half(TF{}, smem + HB, 0, g);
#pragma unroll
  for (int g = 0; g < LX; ++g) load_half(TL{}, smem + 2 * HB, 1, g);
#pragma unroll
  for (int g = 0; g < LW; ++g) load_half(TF{}, smem + 3 * HB, 1, g);
#pragma unroll
  for (int g = 0; g < LX; ++g) load_half(TL{}, smem + 4 * HB, 2, g);
  wait_vmcnt<3 * LX>();  // slice 0 has landed (three halves still in flight)
  barrier_keep_loads();
#pragma unroll
  for (int r = 0; r < TN + TM; ++r) read_frag(XLEAD ? smem : smem + HB, XLEAD ? smem + HB : smem, 0, 0, r);
  // the accumulators were zeroed by VALU writes: two wait states before an
  // MFMA reads them (the assembler statement hides them from the compiler)
  asm volatile("s_nop 1" ::);
  int li = 0, fi = 1;  // buffers of slice kt's lead and other halves
  for (int kt = 0; kt < nk; ++kt) {
    const int ln = li + 2 < 5 ? li + 2 : li - 3, fn = fi + 2 < 5 ? fi + 2 : fi - 3;  // slice kt + 1
    OPS_LDS char* sl = smem + li * HB;
    OPS_LDS char* sf = smem + fi * HB;
    // Past the last slice the loads read zeros into buffers no wave reads
    // any more, and the last slice's look-ahead reads fetch fragments that
    // are never used: one branch-free body keeps every accumulator in one
    // place.
    kstep(B0{}, T{}, F{}, XLEAD ? sl : sf, XLEAD ? sf : sl, 1, sl, sf, kt);
    // slice kt + 1 has landed in every wave (only the lead half of slice
    // kt + 2 stays in flight) and every wave is done reading slice kt, whose
    // buffers take the other half of slice kt + 2 (half 2kt + 5) and the lead
    // half of slice kt + 3 (half 2kt + 6)
    wait_vmcnt<LX>();
    barrier_keep_loads();
    OPS_LDS char* nl = smem + ln * HB;
    OPS_LDS char* nf = smem + fn * HB;
    kstep(B1{}, T{}, T{}, XLEAD ? nl : nf, XLEAD ? nf : nl, 0, sl, sf, kt);
    li = ln;
    fi = fn;
  }
  // The epilogue's reads of the accumulators follow the last MFMA's writes:
  // a 16-pass XDL write needs up to 19 wait states before another
  // instruction reads its result.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::);
  wait_vmem();

  if (tile_part) {
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int r = wm * WM + j * MI + fr;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int c = wn * WN + i * MI + fh * 4;
        *reinterpret_cast<f32x4*>(tile_part + r * BN + c) = agpr_read(acc[i][j]);
      }
    }
    return;
  }
  if (part && tail_cnt == 0) {
    float* pbase = part + (int64_t)split * M * N;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int m = m0 + wm * WM + j * MI + fr;
      if (m - m0 >= m_rows) continue;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int n = n0 + wn * WN + i * MI + fh * 4;
        if (n >= N) continue;
        *reinterpret_cast<f32x4*>(pbase + (int64_t)m * N + n) = agpr_read(acc[i][j]);
      }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm * WM + j * MI + fr;
    if (m - m0 >= m_rows) continue;
    __bf16* yrow = y + (int64_t)m * N;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int n = n0 + wn * WN + i * MI + fh * 4;
      if (n >= N) continue;
      const f32x4 v = agpr_read(acc[i][j]);
      float v0 = v[0], v1 = v[1], v2 = v[2], v3 = v[3];
      if (bias) {
        const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
        v0 += bf_lo(bb[0]);
        v1 += bf_hi(bb[0]);
        v2 += bf_lo(bb[1]);
        v3 += bf_hi(bb[1]);
      }
      *reinterpret_cast<u32x2*>(yrow + n) = u32x2{pack_bf2(v0, v1), pack_bf2(v2, v3)};
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

// y[m][n] = bf16(sum over splits s of part[s][m][n] (in split order) + bias[n]),
// four consecutive elements per thread (N is a multiple of 8).
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int splits,
                                                            const __bf16* __restrict__ bias,
                                                            __bf16* __restrict__ y, int64_t MN, int N) {
  const int64_t n4 = MN / 4;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    f32x4 a = reinterpret_cast<const f32x4*>(part)[i];
    for (int sp = 1; sp < splits; ++sp) a += reinterpret_cast<const f32x4*>(part + (int64_t)sp * MN)[i];
    if (bias) {
      const int n = (int)((i * 4) % N);
      const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
      a[0] += bf_lo(bb[0]);
      a[1] += bf_hi(bb[0]);
      a[2] += bf_lo(bb[1]);
      a[3] += bf_hi(bb[1]);
    }
    reinterpret_cast<u32x2*>(y)[i] = u32x2{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3])};
  }
}

// y of the split tail: tile dp_cnt + t is the sum over splits (in order) of
// its compact partials, plus bias.  Grid (tail_cnt, BM / 16): 16 rows of one
// tile per workgroup, four consecutive columns per thread (N % 8 == 0).
template <int BM, int BN>
__global__ __launch_bounds__(256) void splitk_tile_reduce_kernel(const float* __restrict__ part, int splits,
                                                                 int dp_cnt, int tail_cnt, int M, int N,
                                                                 int tiles_m, int tiles_n, int group_m,
                                                                 const __bf16* __restrict__ bias,
                                                                 __bf16* __restrict__ y) {
  const int t = blockIdx.x;
  int tm, tn;
  tile_coords(dp_cnt + t, tiles_m, tiles_n, group_m, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  constexpr int C4 = BN / 4;
  for (int idx = threadIdx.x; idx < 16 * C4; idx += 256) {
    const int r = blockIdx.y * 16 + idx / C4, c = (idx % C4) * 4;
    const int m = m0 + r, n = n0 + c;
    if (m >= M || n >= N) continue;
    const float* p = part + (int64_t)t * BM * BN + r * BN + c;
    f32x4 a = *reinterpret_cast<const f32x4*>(p);
    for (int sp = 1; sp < splits; ++sp) a += *reinterpret_cast<const f32x4*>(p + (int64_t)sp * tail_cnt * BM * BN);
    if (bias) {
      const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
      a[0] += bf_lo(bb[0]);
      a[1] += bf_hi(bb[0]);
      a[2] += bf_lo(bb[1]);
      a[3] += bf_hi(bb[1]);
    }
    *reinterpret_cast<u32x2*>(y + (int64_t)m * N + n) = u32x2{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3])};
  }
}

// Tile-rows per group of the tile order (tile_coords): as many as keep the
// group's x rows (BM x K bf16 each) within kGroupBytes, so they stay in the
// last-level cache while the group sweeps the tile-columns; at least
// kMinGroupRows, at most all.  The floor matters for long K: an XCD runs 32
// consecutive tiles at once, which with one tile-row per group are 1 x 32
// tiles (all of W's column blocks, re-read by every XCD) and with four are
// 4 x 8.  Measured on the 16384 x 8192 x 28672 down projection: 6590 us with
// one row per group, 5550 with two, 5480 with four, 5640 with eight.
constexpr int64_t kMinGroupRows = 4;
template <class C>
static int tile_group_rows(int64_t tiles_m, int64_t tiles_n, int64_t K) {
  (void)tiles_n;
  const int64_t row_block_bytes = (int64_t)C::BM * K * 2;
  return (int)std::max<int64_t>(1, std::min<int64_t>(tiles_m, std::max(kMinGroupRows, kGroupBytes / row_block_bytes)));
}

// K range of one split: a whole number of BK slices; the number of ranges
// that actually results (at most `splits`).
static int64_t split_chunk(int64_t K, int splits, int BK) { return ((K + splits - 1) / splits + BK - 1) / BK * BK; }
static int split_ranges(int64_t K, int splits, int BK) {
  const int64_t c = split_chunk(K, splits, BK);
  return (int)((K + c - 1) / c);
}

// splits > 1: every tile runs as that many K ranges (fp32 partials [splits, M,
// N] in `part`, then an ordered reduce).  tail_splits > 1: only the tiles of
// the last, partly filled round run split (compact fp32 partial tiles in
// `part`), the other tiles as usual in the same launch.  `part` is the
// caller's workspace, sized by plan_linear.
template <class C, bool XLEAD>
static constexpr auto gemm_kernel() {
  if constexpr (std::is_same<C, CfgW4>::value) return &gemm_bf16_w4_kernel<C, XLEAD>;
  else return &gemm_bf16_kernel<C, false>;
}

// Dynamic LDS of a launch: the four-wave kernel's ring is five half-slices
// (x or W rows of one slice each), the others STAGES whole slices.
template <class C>
static constexpr int gemm_lds_bytes() {
  if constexpr (std::is_same<C, CfgW4>::value) return 5 * C::BM * C::kRowBytes;
  else return C::kLdsBytes;
}

template <class C>
static hipError_t launch_gemm_bf16(const void* x, const void* W, const void* bias, void* y, int64_t M,
                                   int64_t N, int64_t K, hipStream_t s, int splits, int tail_splits, float* part) {
  // More than 64 KB of dynamic LDS per workgroup needs the limit raised once
  // per process (a host-side function attribute, no allocation).
  static const hipError_t attr = [] {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_kernel<C, true>()),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, gemm_lds_bytes<C>());
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_kernel<C, false>()),
                               hipFuncAttributeMaxDynamicSharedMemorySize, gemm_lds_bytes<C>());
  }();
  if (attr != hipSuccess) return attr;
  const int64_t tiles_m = (M + C::BM - 1) / C::BM;
  const int64_t tiles_n = (N + C::BN - 1) / C::BN;
  const int64_t tiles = tiles_m * tiles_n;
  const int group_m = tile_group_rows<C>(tiles_m, tiles_n, K);
  // The four-wave kernel's ring gives two slices of lead to one operand: the
  // one with fewer distinct blocks among the 32 tiles an XCD runs at once (x
  // when a group spans at most 4 tile-rows, i.e. K >= 8192; W for the 8-row
  // groups of K = 4096).  Same-box, flushed: the 8B gate-up 1579 -> 1526 us
  // with W leading, down 769 -> 752 us and the 70B gate-up and down 3-4 %
  // faster with x leading.
  const auto kern = group_m <= 4 ? gemm_kernel<C, true>() : gemm_kernel<C, false>();
  if (tail_splits > 1) {
    const int64_t tail = tiles % kNumCUs, dp = tiles - tail;
    const int64_t kchunk = split_chunk(K, tail_splits, C::BK);
    const int nsplit = split_ranges(K, tail_splits, C::BK);
    hipLaunchKernelGGL(kern, dim3((unsigned)(dp + tail * nsplit)), dim3(C::kThreads), gemm_lds_bytes<C>(),
                       s, static_cast<const __bf16*>(x), static_cast<const __bf16*>(W),
                       static_cast<const __bf16*>(bias), static_cast<__bf16*>(y), (int)M, (int)N, (int)K, group_m,
                       (int)kchunk, part, GroupedGemm{}, (int)dp, (int)tail);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((splitk_tile_reduce_kernel<C::BM, C::BN>), dim3((unsigned)tail, C::BM / 16), dim3(256), 0, s,
                       static_cast<const float*>(part), nsplit, (int)dp, (int)tail, (int)M, (int)N, (int)tiles_m,
                       (int)tiles_n, group_m, static_cast<const __bf16*>(bias), static_cast<__bf16*>(y));
    return hipGetLastError();
  }
  const bool split = splits > 1;
  const int64_t kchunk = split ? split_chunk(K, splits, C::BK) : K;
  const int nsplit = split ? split_ranges(K, splits, C::BK) : 1;
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles * nsplit)), dim3(C::kThreads), gemm_lds_bytes<C>(), s,
                     static_cast<const __bf16*>(x), static_cast<const __bf16*>(W),
                     static_cast<const __bf16*>(bias), static_cast<__bf16*>(y), (int)M, (int)N, (int)K,
                     group_m, (int)kchunk, split ? part : nullptr, GroupedGemm{}, 0, 0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !split) return e;
  return launch_splitk_reduce(part, nsplit, bias, y, M, N, s);
}

hipError_t launch_splitk_reduce(const float* part, int splits, const void* bias, void* y, int64_t M, int64_t N,
                                hipStream_t s) {
  const int64_t MN = M * N;
  const unsigned blocks = (unsigned)std::min<int64_t>(4096, (MN / 4 + 255) / 256);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, part, splits,
                     static_cast<const __bf16*>(bias), static_cast<__bf16*>(y), MN, (int)N);
  return hipGetLastError();
}

// Split-K for small M: when at most half as many 256x128 tiles as CUs exist,
// K is cut into floor(kNumCUs / tiles) ranges (each at least 512 wide), so
// about kNumCUs workgroups run.  (A split that only lifts 129-255 tiles a
// little past the CU count measured slower than no split.)  0: no split.
template <class C>
static int splitk_count(int64_t M, int64_t N, int64_t K) {
  if (M > kSplitKMaxM || K < 1024) return 0;
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  const int64_t s = std::min<int64_t>(kNumCUs / tiles, K / 512);
  return s >= 2 ? (int)s : 0;
}

template <class C>
static hipError_t launch_grouped(const void* x, int64_t x_rows, const void* W, int64_t w_stride, void* y,
                                 int64_t max_rows, int64_t N, int64_t K, int32_t E, const int32_t* gather,
                                 const int32_t* rows, const int32_t* tiles, int32_t swiglu_f, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(gemm_bf16_kernel<C, true>), hipFuncAttributeMaxDynamicSharedMemorySize,
      C::kLdsBytes);
  if (attr != hipSuccess) return attr;
  // at most ceil(rows / BM) + E tile-rows; workgroups past the list's end return
  const int64_t tile_rows = (max_rows + C::BM - 1) / C::BM + E;
  const int64_t tiles_n = (N + C::BN - 1) / C::BN;
  GroupedGemm gg{gather, rows, tiles, E, (int)x_rows, w_stride, swiglu_f};
  hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), dim3((unsigned)(tile_rows * tiles_n)), dim3(C::kThreads),
                     C::kLdsBytes, s, static_cast<const __bf16*>(x), static_cast<const __bf16*>(W), nullptr,
                     static_cast<__bf16*>(y), (int)max_rows, (int)N, (int)K, 1, (int)K, nullptr, gg, 0, 0);
  return hipGetLastError();
}

int32_t grouped_gemm_tile_rows(int64_t rows, int32_t E) {
  // about 96 rows or fewer per expert (decode batches): 64-row tiles, so the
  // matrix cores do not spend most of a 256-row tile on padding
  return rows <= (int64_t)96 * E ? CfgRow64::BM : CfgBig8::BM;
}

hipError_t launch_gemm_grouped(const void* x, int64_t x_rows, const void* W, int64_t w_stride, void* y,
                               int64_t max_rows, int64_t N, int64_t K, int32_t E, int32_t tile_rows,
                               const int32_t* gather, const int32_t* rows, const int32_t* tiles, int32_t swiglu_f,
                               hipStream_t s) {
  if (tile_rows == CfgRow64::BM)
    return launch_grouped<CfgRow64>(x, x_rows, W, w_stride, y, max_rows, N, K, E, gather, rows, tiles, swiglu_f, s);
  return launch_grouped<CfgBig8>(x, x_rows, W, w_stride, y, max_rows, N, K, E, gather, rows, tiles, swiglu_f, s);
}

// The tiled configurations a plan can name.
enum TileCfg { kCfgBig8 = 0, kCfgT192 = 1, kCfgMid = 2, kCfgSk64 = 3, kCfgSk128 = 4, kCfgW4 = 5 };

template <class C>
static size_t split_bytes(int64_t M, int64_t N, int64_t K, int splits) {
  return (size_t)split_ranges(K, splits, C::BK) * M * N * sizeof(float);
}

template <class C>
static size_t tail_bytes(int64_t M, int64_t N, int64_t K, int tail_splits) {
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  return (size_t)split_ranges(K, tail_splits, C::BK) * (tiles % kNumCUs) * C::BM * C::BN * sizeof(float);
}

// One rule for the path of a linear, shared by the workspace query and the
// launch.  split_ok == false (no caller workspace) plans only paths that need
// none: the small-M kernel or unsplit tiles.
LinearPlan plan_linear(int64_t M, int64_t N, int64_t K, bool bf16, bool split_ok) {
  LinearPlan p{};
  if (!bf16) { p.path = LinearPlan::kF32; return p; }
  const int32_t force_tile = tuning(OPSCALE_TUNE_GEMM_TILE);
  const int32_t skinny = tuning(OPSCALE_TUNE_GEMM_SKINNY);
  p.path = LinearPlan::kTiled;
  // Decode-sized M: the weights dominate and large tiles would leave most CUs
  // idle.  The small-M kernel reduces its K split in LDS and needs no
  // workspace.
  if (force_tile < 0 && skinny != 0 &&
      (skinny == 1 ? skinny_linear_supported(M, N, K) : skinny_linear_preferred(M, N, K))) {
    p.path = LinearPlan::kSkinny;
    return p;
  }
  // Decode batches of 33-128 rows with K up to 8192: the weight-streaming
  // kernel, its K split (if any) through the workspace.  Measured cold on
  // the 8B-layer projections it is 3-13 % faster there than the split-K tiles
  // (QKV, O, gate-up at M = 64 and 128); at 192-256 rows and for the
  // 14336-wide down projection the tiles below are faster.
  const int32_t dec = tuning(OPSCALE_TUNE_GEMM_DECODE);
  if (force_tile < 0 && dec != 0 && decode_linear_supported(M, N, K) &&
      (dec == 1 || (M > 32 && M <= 128 && K <= 8192))) {
    const int ds = tuning(OPSCALE_TUNE_GEMM_SPLITK) == 0 ? 1 : decode_linear_splits(M, N, K);
    if (ds <= 1 || split_ok) {
      p.path = LinearPlan::kDecode;
      p.splits = ds;
      p.ws_bytes = ds > 1 ? decode_linear_ws_bytes(M, N, K) : 0;
      return p;
    }
  }
  // Otherwise decode-sized M splits K over workgroups (fp32 partials in the
  // workspace, summed in split order by a second kernel).  Tile rows follow
  // M: 64 up to 64 rows (the matrix cores work on little padding), 128 up to
  // 256; larger M takes 256 rows with 256 or 128 columns, whichever gives
  // more workgroups (ties: 256, which re-reads x half as often).
  if (force_tile < 0 && split_ok && tuning(OPSCALE_TUNE_GEMM_SPLITK) != 0) {
    if (M <= 64) {
      p.splits = splitk_count<CfgSk64>(M, N, K);
      p.cfg = kCfgSk64;
      if (p.splits > 1) { p.ws_bytes = split_bytes<CfgSk64>(M, N, K, p.splits); return p; }
    } else if (M <= 256) {
      p.splits = splitk_count<CfgSk128>(M, N, K);
      p.cfg = kCfgSk128;
      if (p.splits > 1) { p.ws_bytes = split_bytes<CfgSk128>(M, N, K, p.splits); return p; }
    } else {
      const int s_wide = splitk_count<CfgBig8>(M, N, K), s_mid = splitk_count<CfgMid>(M, N, K);
      const int64_t w_wide = (int64_t)s_wide * ((N + 255) / 256), w_mid = (int64_t)s_mid * ((N + 127) / 128);
      if (w_wide >= w_mid && s_wide > 1) {
        p.cfg = kCfgW4; p.splits = s_wide; p.ws_bytes = split_bytes<CfgW4>(M, N, K, s_wide); return p;
      }
      if (s_mid > 1) { p.cfg = kCfgMid; p.splits = s_mid; p.ws_bytes = split_bytes<CfgMid>(M, N, K, s_mid); return p; }
    }
    p.splits = 0;
  }
  // 129-256 rows whose 128-row tiles already fill more than half the GPU
  // (the gate-up projection of a 256-sequence decode batch: 224 tiles) run
  // unsplit as 128-row tiles: their 3-stage ring keeps two weight slices per
  // CU in flight.
  if (force_tile < 0 && M > 128 && M <= 256 && K >= 1024 &&
      2 * ((N + CfgSk128::BN - 1) / CfgSk128::BN) > kNumCUs / 2) {
    p.cfg = kCfgSk128;
    return p;
  }
  // A last round at most half full runs split over K: 2-4 ranges per tile
  // (at most one workgroup per CU in all), each at least 8 slices long.
  const bool tail_ok = split_ok && tuning(OPSCALE_TUNE_GEMM_TAIL) != 0;
  auto tail_splits = [&](int64_t tiles) {
    const int64_t tail = tiles % kNumCUs;
    if (!tail_ok || tiles <= kNumCUs || tail == 0 || tail * 2 > kNumCUs) return 0;
    const int ts = (int)std::min<int64_t>(std::min<int64_t>(4, kNumCUs / tail), K / (8 * 64));
    return ts < 2 ? 0 : ts;
  };
  // One workgroup per CU at a time, so a launch runs in full rounds plus a
  // last one (a split last round counts as 1 / splits of a round).  Pick the
  // tile whose rounds x tile area x relative per-element cost is smallest:
  // 256x256 moves the fewest operand bytes per flop; 192x256 (measured about
  // 17 % more time per element) and 256x128 (about 60 % more) fill the last
  // round better when 256x256 would leave it mostly idle.
  struct Choice { int bm, bn; double cost; };
  static constexpr Choice choices[] = {{256, 256, 1.0}, {192, 256, 1.17}, {256, 128, 1.6}};
  int best = 0;
  if (force_tile >= 0 && force_tile <= 3) {
    best = force_tile == 3 ? 0 : force_tile;
  } else {
    double best_t = 0;
    for (int c = 0; c < 3; ++c) {
      const int64_t tiles = ((M + choices[c].bm - 1) / choices[c].bm) * ((N + choices[c].bn - 1) / choices[c].bn);
      const int ts = tail_splits(tiles);
      const double rounds = (double)(tiles / kNumCUs) + (tiles % kNumCUs == 0 ? 0.0 : ts ? 1.0 / ts : 1.0);
      const double t = rounds * choices[c].bm * choices[c].bn * choices[c].cost;
      if (c == 0 || t < best_t) { best = c; best_t = t; }
    }
  }
  p.cfg = best == 0 ? (force_tile == 3 ? kCfgBig8 : kCfgW4) : best == 1 ? kCfgT192 : kCfgMid;
  p.tail_splits = tail_splits(((M + choices[best].bm - 1) / choices[best].bm) *
                              ((N + choices[best].bn - 1) / choices[best].bn));
  if (p.tail_splits > 1)
    p.ws_bytes = p.cfg == kCfgBig8 || p.cfg == kCfgW4 ? tail_bytes<CfgBig8>(M, N, K, p.tail_splits)
                 : p.cfg == kCfgT192 ? tail_bytes<CfgT192>(M, N, K, p.tail_splits)
                                     : tail_bytes<CfgMid>(M, N, K, p.tail_splits);
  return p;
}

hipError_t launch_linear(const LinearPlan& p, const void* x, const void* W, const void* bias, void* y, int64_t M,
                         int64_t N, int64_t K, void* ws, hipStream_t s) {
  float* part = static_cast<float*>(ws);
  switch (p.path) {
    case LinearPlan::kSkinny:
      return launch_linear_skinny(x, W, bias, y, M, N, K, s);
    case LinearPlan::kDecode:
      return launch_linear_decode(x, W, bias, y, M, N, K, p.splits, ws, s);
    case LinearPlan::kTiled:
      switch (p.cfg) {
        case kCfgBig8: return launch_gemm_bf16<CfgBig8>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
        case kCfgW4: return launch_gemm_bf16<CfgW4>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
        case kCfgT192: return launch_gemm_bf16<CfgT192>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
        case kCfgMid: return launch_gemm_bf16<CfgMid>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
        case kCfgSk64: return launch_gemm_bf16<CfgSk64>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
        default: return launch_gemm_bf16<CfgSk128>(x, W, bias, y, M, N, K, s, p.splits, p.tail_splits, part);
      }
    default: break;
  }
  const dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, static_cast<const float*>(x),
                     static_cast<const float*>(W), static_cast<const float*>(bias),
                     static_cast<float*>(y), (int)M, (int)N, (int)K);
  return hipGetLastError();
}

}  // namespace opscale
