// Device helpers shared by the gfx950 kernels of libopscale.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace opscale {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define OPS_LDS __attribute__((address_space(3)))

// 0x00020000: raw buffer, 32-bit dword format, no swizzle (the CDNA value).
constexpr int kBufferFlags = 0x00020000;
// Any voffset >= num_records reads as zero; used to mask a lane's load.
constexpr uint32_t kOobOffset = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferFlags);
}

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0);
}

// 16 bytes per lane straight into LDS at lds_wave_base + lane * 16.  POLICY
// is the instruction's cache-policy field; kNoL1 (sc0) keeps the line out of
// the CU's L1, for data each CU reads once (it still allocates in L2).
constexpr int kNoL1 = 1;
template <int POLICY = 0>
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t r, OPS_LDS void* lds_wave_base,
                                                  uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_wave_base, 16, voff, 0, 0, POLICY);
}

// 16 bytes per lane from a 64-bit global address into LDS at lds_wave_base +
// lane * 16 (global_load_lds_dwordx4).
__device__ __forceinline__ void global_load16_lds(const void* gptr, OPS_LDS void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(gptr, lds_wave_base, 16, 0, 0);
}

// The same with the nontemporal hint (data read once, not kept in the caches).
__device__ __forceinline__ void global_load16_lds_nt(const void* gptr, OPS_LDS void* lds_wave_base) {
  constexpr int kNontemporal = 2;  // cache-policy bit NT on gfx950
  __builtin_amdgcn_global_load_lds(gptr, lds_wave_base, 16, 0, kNontemporal);
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Two floats -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Integer sum / max over a fully active wave, returned wave-uniform.  The
// 16-lane rows reduce with DPP moves (quad_perm [1,0,3,2], quad_perm
// [2,3,0,1], row_half_mirror, row_mirror: after the four steps every lane of
// a row holds the row's result), the four rows through readlane, so the chain
// never touches LDS (unlike a shuffle, which is a ds_bpermute).
__device__ __forceinline__ int row_dpp_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xf, 0xf, false);
  return v;
}
__device__ __forceinline__ int row_dpp_max(int v) {
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xf, 0xf, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xf, 0xf, false));
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
  v = row_dpp_sum(v);
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) + __builtin_amdgcn_readlane(v, 32) +
         __builtin_amdgcn_readlane(v, 48);
}
__device__ __forceinline__ int wave_max_i(int v) {
  v = row_dpp_max(v);
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}
// The same DPP row reductions for floats (fixed order: deterministic).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_max_f(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x141>(v));
  v = fmaxf(v, dpp_f<0x140>(v));
  auto lane = [&](int l) { return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l)); };
  return fmaxf(fmaxf(lane(0), lane(16)), fmaxf(lane(32), lane(48)));
}
__device__ __forceinline__ float wave_sum_f(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  auto lane = [&](int l) { return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l)); };
  return (lane(0) + lane(16)) + (lane(32) + lane(48));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wait for every outstanding vector-memory operation of this wave (including
// buffer loads into LDS) before a barrier makes their data visible.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0); }

// s_waitcnt constraining only the vector-memory counter to <= N (gfx9
// encoding: vmcnt in bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt_le() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for rings filled by LDS DMA (buffer_load ... lds): this
// wave's LDS reads are complete and the compiler moves no memory access across
// it, but its LDS DMA loads stay in flight.  __syncthreads() would also wait
// for those (a workgroup fence counts an LDS DMA load as an LDS write), which
// drains a multi-stage ring at every barrier; the caller instead waits for the
// slice it needs with wait_vmcnt_le<N>() first.
__device__ __forceinline__ void barrier_keep_loads() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Block id -> tile id such that the consecutive tile ids land on one XCD.
// Workgroups are dealt round-robin to the 8 XCDs, so block b runs on XCD
// b % 8; giving each XCD a contiguous range of tiles keeps neighbouring tiles
// (which share operand rows) in the same 4 MB L2.  A bijection for any count.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t total) {
  constexpr uint32_t kXcd = 8;
  const uint32_t per = total / kXcd, rem = total % kXcd;
  const uint32_t x = bid % kXcd, i = bid / kXcd;
  const uint32_t start = x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per;
  return start + i;
}

}  // namespace opscale
