// Internal declarations shared by the host library and the HIP kernels.
//
// Internal cell order.  Each dataset b keeps only its S_b active cell columns.  Active
// columns of all datasets are numbered globally, dataset-major: column g belongs to dataset
// col_ds[g] and is native cell column col_c[g].  Active cell p is (column g = p / R, row
// r = p % R), so every column is R consecutive cells — the item axis reads contiguous rows —
// and the cells of row (b, r) are p = (col0[b] + k) * R + r, k in [0, S_b).
//
// Item-axis Q/K/V are stored head-major per column: [g][head][R][d].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tfm {

// Per-dataset metadata on the device.
struct DsInfo {
  int32_t n_train;  // train-prefix length
  int32_t col0;     // first global active column of the dataset
  int32_t S;        // number of active cell columns
  int32_t pad;
};

// Everything a kernel needs to map internal indices to the native [B][R][S][E] layout.
struct Geo {
  int32_t B, R, S, E, heads, d, H;
  int32_t NC;              // total active columns
  int64_t N;               // total active cells = NC * R
  const DsInfo* ds;        // [B]
  const int32_t* col_ds;   // [NC] dataset of each active column
  const int32_t* col_c;    // [NC] native cell column of each active column
  const int32_t* colmap;   // [B*S] native (b, c) -> global active column, or -1
  // Per-column copies of the above that a kernel reads with one load instead of a dependent
  // pair: the native cell index of the column's row 0, (col_ds * R) * S + col_c, and the
  // train-prefix length of the column's dataset.
  const int64_t* col_cell0;  // [NC]
  const int32_t* col_ntr;    // [NC]
  int32_t nmax;              // longest train prefix over the datasets
};

// A subset of the active columns in a chosen order: column cols[i] for i < count; cols null
// means every column in order (count = NC).
struct ColList {
  const int32_t* cols;
  int32_t count;
};

__host__ __device__ inline int64_t native_cell(const Geo& g, int64_t p) {
  int64_t col = p / g.R;
  int64_t r = p - col * g.R;
  return g.col_cell0[col] + r * g.S;
}

// bfloat16 storage as raw 16-bit patterns; round to nearest even on store.
typedef uint16_t bf16;

__device__ __forceinline__ float ld(const float* p) { return *p; }
__device__ __forceinline__ float ld(const bf16* p) {
  return __uint_as_float(((uint32_t)(*p)) << 16);
}
__device__ __forceinline__ void st(float* p, float v) { *p = v; }
__device__ __forceinline__ uint16_t f2bf(float v) {
  uint32_t u = __float_as_uint(v);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ void st(bf16* p, float v) { *p = f2bf(v); }

// Launch helpers return hipError_t of the launch.
#define TFM_BLOCK 256

}  // namespace tfm
