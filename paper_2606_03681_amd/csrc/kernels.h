// Host-side launchers of the HIP kernels.  Each returns the hipError_t of its launch(es).
#pragma once

#include "common.h"

namespace tfm {

// ---- metadata -------------------------------------------------------------------------------
// Copies `count` int32 values from host memory into device memory at `dst` through kernel
// arguments (stream-ordered, no host synchronisation, host memory free to reuse at return).
hipError_t launch_upload(const int32_t* host, int64_t count, int32_t* dst, hipStream_t s);
// Expands the per-dataset blob {n_train, col0, S_b, mask words...} into DsInfo and the
// column maps of Geo.
hipError_t launch_expand_meta(const int32_t* blob, int B, int R, int S, int words, DsInfo* ds,
                              int32_t* col_ds, int32_t* col_c, int32_t* colmap,
                              int64_t* col_cell0, int32_t* col_ntr, hipStream_t s);

// ---- data movement between the native [B][R][S][E] layout and active cells ------------------
template <class T>
hipError_t launch_gather(const Geo& g, const T* native, T* cells, hipStream_t s);
// dst_native = a (+ b) at active cells, 0 at inactive cells.  b may be null.
template <class T>
hipError_t launch_scatter(const Geo& g, const T* a, const T* b, T* native, hipStream_t s);

// ---- simple (VALU, fp32 arithmetic) kernels, any storage type ------------------------------
// out[m, j] = sum_i A[m*lda + i] * w[j*wsj + i*wsi] + bias[j]  (bias may be null)
template <class TA, class TO>
hipError_t launch_linear(int64_t M, int Nout, int K, const TA* A, int64_t lda, const float* w,
                         int64_t wsj, int64_t wsi, const float* bias, TO* out, int64_t ldo,
                         hipStream_t s);
// Item-axis Q|K|V projection written head-major: q/k/v[((col*heads+h)*R + r)*d + j];
// K and V only for train rows.
template <class T>
hipError_t launch_linear_item_qkv(const Geo& g, const T* A, const float* w, const float* bias,
                                  T* q, T* k, T* v, hipStream_t s);
// partial[z][j][i] = sum over rows m of chunk z of dY[m*ldy + j] * X[m*ldx + i]
template <class T>
hipError_t launch_wgrad(int64_t M, int Nj, int Ki, const T* dY, int64_t ldy, const T* X,
                        int64_t ldx, int64_t chunk, float* partial, hipStream_t s);
// partial[z][j] = sum over rows m of chunk z of A[m*lda+j] (* B[m*ldb+j] if B non-null)
template <class T>
hipError_t launch_colsum(int64_t M, int Nj, const T* A, int64_t lda, const T* B, int64_t ldb,
                         int64_t chunk, float* partial, hipStream_t s);
// grad[i] = (accumulate ? grad[i] : 0) + sum_z partial[z*count + i], z ascending
hipError_t launch_reduce_partials(int Z, int64_t count, const float* partial, float* grad,
                                  int accumulate, hipStream_t s);

// h = LN(a + b) (b may be null); xhat and rstd saved for the backward pass.
template <class T>
hipError_t launch_add_ln(int64_t N, int E, const T* a, const T* b, const float* gamma,
                         const float* beta, T* h, T* xhat, float* rstd, hipStream_t s);
// du = LN'(dy) with dy = dya (+ dyb); dysum (nullable) receives dy.
template <class T>
hipError_t launch_ln_bwd(int64_t N, int E, const T* dya, const T* dyb, const T* xhat,
                         const float* rstd, const float* gamma, T* du, T* dysum, hipStream_t s);
template <class T>
hipError_t launch_gelu(int64_t count, const T* g, T* u, hipStream_t s);
// du <- du * GELU'(g), in place
template <class T>
hipError_t launch_gelu_bwd(int64_t count, const T* g, T* du, hipStream_t s);

template <class T>
hipError_t launch_feat_attn_fwd_simple(const Geo& g, const T* qkv, T* o, float* lse,
                                       hipStream_t s);
template <class T>
hipError_t launch_feat_attn_bwd_simple(const Geo& g, const T* qkv, const T* o, const T* dout,
                                       const float* lse, T* dqkv, hipStream_t s);
template <class T>
hipError_t launch_item_attn_fwd_simple(const Geo& g, const T* q, const T* k, const T* v, T* o,
                                       float* lse, hipStream_t s);
// dq/dk/dv head-major; D is scratch [NC*heads*R]
template <class T>
hipError_t launch_item_attn_bwd_simple(const Geo& g, const T* q, const T* k, const T* v,
                                       const T* o, const T* dout, const float* lse, float* D,
                                       T* dq, T* dk, T* dv, hipStream_t s);
// cell-major [N][3E] from head-major dq/dk/dv, with 0 for K/V of non-train rows
template <class T>
hipError_t launch_item_dqkv_to_cells(const Geo& g, const T* dq, const T* dk, const T* dv,
                                     T* dqkv, hipStream_t s);

}  // namespace tfm
