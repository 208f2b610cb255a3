// MFMA attention kernels of the layer: launch interfaces.
#pragma once

#include "common.h"

namespace tfm {

// Item-axis attention forward.  q head-major [col][head][R][d], k/v head-major
// [col][head][kR][d] valid for the first n_train rows (kR = R when kR <= 0; a larger kR lets the
// queries of one call read keys and values kept from another call with more rows), o
// cell-major [cell][E], lse [col][head][R] (natural log of the softmax denominator including
// the 1/sqrt(d) scale).
hipError_t launch_item_attn_fwd(const Geo& g, const bf16* q, const bf16* k, const bf16* v,
                                bf16* o, float* lse, hipStream_t s, int kR = 0);

// Item-axis attention backward: dq, dk, dv head-major (dk, dv for train rows only).
// Backward in two launches, dQ first: it also writes Dbuf ([problem][R] float32) with
// D = rowsum(dO o O) per query row, which the dK/dV launch reads.
// Both run over the problems of the columns in cl (every column when cl.cols is null).
hipError_t launch_item_attn_dq(const Geo& g, const ColList& cl, const bf16* q, const bf16* k,
                               const bf16* v, const bf16* o, const bf16* dout, const float* lse,
                               float* Dbuf, bf16* dq, hipStream_t s);
hipError_t launch_item_attn_dkdv(const Geo& g, const ColList& cl, const bf16* q, const bf16* k,
                                 const bf16* v, const bf16* o, const bf16* dout,
                                 const float* lse, const float* Dbuf, bf16* dk, bf16* dv,
                                 hipStream_t s);

// The same backward in one launch for train prefixes of at most 768 rows at d in {16, 32}
// (item_attn_bwd_fused_ok): one workgroup per (column, head) problem of the columns in cl
// computes P and dS once per score and writes dq, dk and dv; nmax is the longest train prefix
// among those columns.
bool item_attn_bwd_fused_ok(const Geo& g, int nmax);
int item_attn_bwd_fused_max_rows(int d);
hipError_t launch_item_attn_bwd_fused(const Geo& g, const ColList& cl, int nmax, const bf16* q,
                                      const bf16* k, const bf16* v, const bf16* o,
                                      const bf16* dout, const float* lse, bf16* dq, bf16* dk,
                                      bf16* dv, hipStream_t s);

// Feature-axis attention (cells of a row, per head).  qkv cell-major [cell][3E]; o, dout
// cell-major [cell][E]; lse [cell][heads]; dqkv cell-major [cell][3E].  Requires
// feat_attn_mfma_ok(g) (at most 128 active cells per row, 32-bit row offsets).
bool feat_attn_mfma_ok(const Geo& g);
hipError_t launch_feat_attn_fwd(const Geo& g, const bf16* qkv, bf16* o, float* lse,
                                hipStream_t s);
hipError_t launch_feat_attn_bwd(const Geo& g, const bf16* qkv, const bf16* o, const bf16* dout,
                                const float* lse, bf16* dqkv, hipStream_t s);

}  // namespace tfm
