// CDNA4 (gfx950) matrix-core helpers shared by the MFMA kernels.
//
// v_mfma_f32_16x16x32_bf16 operand layout (64-lane wave, g = lane / 16, c = lane % 16):
//   A (16 x 32): lane holds A[c][8g .. 8g+7]        (8 bf16, 16 bytes)
//   B (32 x 16): lane holds B[8g .. 8g+7][c]        (8 bf16, 16 bytes)
//   D (16 x 16): lane holds D[4g .. 4g+3][c]        (4 f32)
// Any permutation of the 32 k positions that is applied to A and B alike gives the same
// product, which the attention kernels use to feed a D tile back in as an operand.
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

namespace tfm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

// 16-byte loads/stores of 8 bf16 values.
__device__ __forceinline__ bf16x8 ld8(const bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ uint4 ldu4(const bf16* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void stu4(bf16* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float(((uint32_t)u) << 16); }

// LDS transpose read (ds_read_b64_tr_b16).  Every lane names an 8-byte LDS address (four
// bf16); within each group of 16 lanes, lane i receives as its element j the element i % 4 of
// the four named by lane 4j + i / 4.  So if lane L of a group names row L / 4, columns
// c0 + 4 (L % 4) .. +3 of a row-major tile, lane i receives column c0 + i of rows 0..3: a
// 4-deep slice of an MFMA operand whose contraction index runs down the tile's rows.
__device__ __forceinline__ bf16x4 lds_read_tr16(const bf16* p) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}

// MFMA fragment whose k positions run down the rows of a row-major LDS tile T (row stride ls
// elements): lane (g, c) receives column c0 + c of rows 4g .. 4g+3 (slots 0-3) and
// 16 + 4g .. 16 + 4g + 3 (slots 4-7).  That is the k order of two 16-row D tiles packed
// side by side, so an S tile can meet the transposed operand it multiplies.  Conflict-free
// when ls * 2 bytes is an odd multiple of 32.
__device__ __forceinline__ bf16x8 ld_tr8(const bf16* T, int ls, int c0, int lane) {
  const bf16* p = T + (lane >> 2) * ls + c0 + 4 * (lane & 3);
  const bf16x4 lo = lds_read_tr16(p), hi = lds_read_tr16(p + 16 * ls);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Index of the calling wave in its workgroup, as a wave-uniform (scalar) value: values derived
// from it (a wave's row, problem, key range) then stay in SGPRs and branches on them are scalar.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Round-to-nearest-even pack of two floats into two bf16 (low half = a): v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  return *reinterpret_cast<uint32_t*>(&r);
}

// One bf16 from a float (round to nearest even) through the hardware convert.
__device__ __forceinline__ uint16_t to_bf16(float a) { return (uint16_t)(pack2(a, 0.f) & 0xffffu); }

// 2^x on the transcendental unit (v_exp_f32), without the library's range handling; the
// callers pass arguments <= 0 whose results below the float range may flush to 0.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Buffer resources: 32-bit offsets from an SGPR descriptor; loads at offsets >= bytes return 0
// (the hardware range check of raw buffers), which the kernels use for ragged tails.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ __forceinline__ uint4 bload16(rsrc_t r, uint32_t off) {
  u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 bload8(rsrc_t r, uint32_t off) {
  u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return make_uint2(v.x, v.y);
}
__device__ __forceinline__ float bloadf(rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// 16 bytes per lane from global memory into LDS at lds_dst + 16 * lane (lds_dst wave-uniform).
// Issued through inline assembly so that the compiler does not add its own conservative
// vmcnt waits before later LDS reads: the pipeline waits for these loads explicitly.
__device__ __forceinline__ void lds_dma16(const void* src, bf16* lds_dst) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_dst);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(m0v), "v"(src)
               : "memory", "m0");
}

// The same DMA from a wave-uniform base address (SGPRs) plus a per-lane byte offset: lane L's 16
// bytes come from sbase + voff and land at lds_dst + 16 * L.  One VGPR of address per lane.
__device__ __forceinline__ void lds_dma16_s(const void* sbase, uint32_t voff, bf16* lds_dst) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_dst);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(m0v), "v"(voff), "s"(sbase)
               : "memory", "m0");
}

// Workgroup barrier that waits only for this wave's LDS traffic (lgkmcnt), not for global
// loads still in flight, so that prefetches issued before it keep overlapping compute.
// The memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Element j (0..7) of 8 bf16 values held in a uint4, as raw bits (j must be a constant after
// unrolling; no memory round trip).
__device__ __forceinline__ uint16_t u4_elem(const uint4& u, int j) {
  const uint32_t w = j < 2 ? u.x : (j < 4 ? u.y : (j < 6 ? u.z : u.w));
  return (uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu));
}

// Cross-lane sums and maxima that stay in the VALU (no LDS permute).  Within a 16-lane row:
// DPP moves pair lanes i ^ 1 and i ^ 2 (quad permutes), then the half-row mirror and the row
// mirror pair the same groups of four and eight lanes as i ^ 4 and i ^ 8 would.  Across the
// four rows: the row swaps of gfx950 (rows 0 <-> 1 and 2 <-> 3, then the two halves).  Every
// lane of the group ends with the same value, added in the same tree as an xor butterfly.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
// Sum over the 16 lanes of the lane's row (lanes sharing lane / 16).
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  return v;
}
// Sum over the 32 lanes of the lane's half-wave (lanes sharing lane / 32).
__device__ __forceinline__ float half32_sum(float v) {
  v = row16_sum(v);
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
// Sum and maximum over the 4 lanes that share lane % 16 (one per row).
__device__ __forceinline__ float rows4_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float rows4_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float wave_reduce_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace tfm
