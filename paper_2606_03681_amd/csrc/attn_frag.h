// Per-head MFMA fragments for the attention kernels: products over the head dimension d,
// A (16 rows x d) times B (d x 16 columns), for d in {16, 32, 64}.
//
// Lane (g = lane / 16, c = lane % 16) holds row (or column) c:
//   d = 16: values 4g .. 4g+3                    (v_mfma_f32_16x16x16_bf16)
//   d = 32: values 8g .. 8g+7                    (v_mfma_f32_16x16x32_bf16)
//   d = 64: values 8g .. 8g+7 and 32+8g .. 32+8g+7 (two 16x16x32 products accumulated)
#pragma once

#include "mfma.h"

namespace tfm {

typedef short s16x4 __attribute__((ext_vector_type(4)));

template <int D>
struct HF;

template <>
struct HF<16> {
  typedef s16x4 frag;
  static constexpr int EPL = 4;  // values per lane
  static __device__ __forceinline__ frag lds(const bf16* row, int lg) {
    return *reinterpret_cast<const s16x4*>(row + lg * 4);
  }
  static __device__ __forceinline__ frag glob(const bf16* row, int lg) { return lds(row, lg); }
  static __device__ __forceinline__ frag buf(rsrc_t r, uint32_t rowbyte, int lg) {
    uint2 u = bload8(r, rowbyte + lg * 8);
    return *reinterpret_cast<s16x4*>(&u);
  }
  static __device__ __forceinline__ frag zero() { return frag{}; }
  static __device__ __forceinline__ f32x4 mma(const frag& a, const frag& b,
                                             const f32x4& c = zero4()) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t elem(const frag& f, int j) {
    return (uint16_t)f[j];
  }
  static __device__ __forceinline__ int dim(int lg, int j) { return lg * 4 + j; }
};

template <>
struct HF<32> {
  typedef bf16x8 frag;
  static constexpr int EPL = 8;
  static __device__ __forceinline__ frag lds(const bf16* row, int lg) { return ld8(row + lg * 8); }
  static __device__ __forceinline__ frag glob(const bf16* row, int lg) { return lds(row, lg); }
  static __device__ __forceinline__ frag buf(rsrc_t r, uint32_t rowbyte, int lg) {
    uint4 u = bload16(r, rowbyte + lg * 16);
    return *reinterpret_cast<bf16x8*>(&u);
  }
  static __device__ __forceinline__ frag zero() { return frag{}; }
  static __device__ __forceinline__ f32x4 mma(const frag& a, const frag& b,
                                             const f32x4& c = zero4()) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t elem(const frag& f, int j) {
    return u4_elem(*reinterpret_cast<const uint4*>(&f), j);
  }
  static __device__ __forceinline__ int dim(int lg, int j) { return lg * 8 + j; }
};

template <>
struct HF<64> {
  struct frag {
    bf16x8 lo, hi;
  };
  static constexpr int EPL = 16;
  static __device__ __forceinline__ frag lds(const bf16* row, int lg) {
    return frag{ld8(row + lg * 8), ld8(row + 32 + lg * 8)};
  }
  static __device__ __forceinline__ frag glob(const bf16* row, int lg) { return lds(row, lg); }
  static __device__ __forceinline__ frag buf(rsrc_t r, uint32_t rowbyte, int lg) {
    uint4 a = bload16(r, rowbyte + lg * 16), b = bload16(r, rowbyte + 64 + lg * 16);
    return frag{*reinterpret_cast<bf16x8*>(&a), *reinterpret_cast<bf16x8*>(&b)};
  }
  static __device__ __forceinline__ frag zero() { return frag{}; }
  static __device__ __forceinline__ f32x4 mma(const frag& a, const frag& b,
                                             const f32x4& c = zero4()) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        a.hi, b.hi, __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.lo, b.lo, c, 0, 0, 0), 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t elem(const frag& f, int j) {
    return j < 8 ? u4_elem(*reinterpret_cast<const uint4*>(&f.lo), j)
                 : u4_elem(*reinterpret_cast<const uint4*>(&f.hi), j - 8);
  }
  static __device__ __forceinline__ int dim(int lg, int j) {
    return j < 8 ? lg * 8 + j : 32 + lg * 8 + (j - 8);
  }
};

// An empty use of a fragment's registers: the compiler waits for the loads that fill them here,
// so no wait for them is left pending at the head of a later loop.
template <int D>
__device__ __forceinline__ void hf_touch(const typename HF<D>::frag& f) {
  if constexpr (D == 64)
    asm volatile("" ::"v"(f.lo), "v"(f.hi));
  else
    asm volatile("" ::"v"(f));
}

// Sum over the lane's values of a * b (one lane's share of a row dot product).
template <int D>
__device__ __forceinline__ float hf_dot(const typename HF<D>::frag& a,
                                        const typename HF<D>::frag& b) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < HF<D>::EPL; ++j) s = fmaf(bf2f(HF<D>::elem(a, j)), bf2f(HF<D>::elem(b, j)), s);
  return s;
}

// LDS row stride (elements) of row-major [key][d] tiles read with ld_tr8: an odd multiple of
// 32 bytes that holds d values.
template <int D>
constexpr int tr_stride() {
  return D <= 32 ? 48 : 80;
}

// LDS tiles of 64-byte rows (32 bf16: d = 32, or 32 queries): the two 16-byte halves of each
// 32-byte chunk and the two chunks are swapped by bits 1 and 2 of the row.  Measured on this
// LDS, that makes 16-byte row accesses (16 rows, one column, per instruction) and transposed
// reads (8 rows of one 32-byte chunk per half-wave) free of bank conflicts, where padded rows
// serve one of the two at best.  Returns the physical byte offset within row r.
__device__ __forceinline__ int row64_swz(int r, int byte) {
  return byte ^ (((r >> 1) & 1) << 4) ^ (((r >> 2) & 1) << 5);
}

// Transposed read (ds_read_b64_tr_b16) of a row64 tile: off is the lane's byte offset of row
// lane / 4 (row64_swz applied; unchanged by multiples of 8 rows), T the tile's first row of the
// 32-row step.  Lane (g, c) receives the column the offset names, of rows {4g .. 4g+3} (slots
// 0-3) and 16 + {4g .. 4g+3} (slots 4-7).
__device__ __forceinline__ bf16x8 tr8_row64(const bf16* T, int off) {
  const bf16* p = T + off / 2;
  const bf16x4 lo = lds_read_tr16(p), hi = lds_read_tr16(p + 16 * 32);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

}  // namespace tfm
