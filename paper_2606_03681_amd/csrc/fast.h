// MFMA (bfloat16) kernels of the layer: launch interfaces.
#pragma once

#include <stddef.h>

#include "common.h"

namespace tfm {

// Where rows of an operand live: compact active cells (row m at m * ld) or the native
// [B][R][S][E] tensor (row m at native_cell(m) * E).
// ROWS_ITEM_HM: the item-axis Q|K|V gradients, head-major [col][head][R][d] in three arrays
// (Q, K, V); row m = cell, column k in [0, 3E); K and V read as 0 at non-train rows.
enum { ROWS_COMPACT = 0, ROWS_NATIVE = 1, ROWS_ITEM_HM = 2 };

// Element offset of (cell m, column k) in the head-major item Q|K|V arrays; part receives
// 0 (Q), 1 (K) or 2 (V); returns -1 where K/V do not exist (non-train rows).
__device__ __forceinline__ int64_t item_hm_offset(const Geo& g, int64_t col, int r, int k,
                                                  int* part) {
  const int p = k / g.E, within = k - p * g.E;
  const int head = within / g.d, j = within - head * g.d;
  *part = p;
  if (p > 0 && r >= g.col_ntr[col]) return -1;
  return ((col * g.heads + head) * g.R + r) * g.d + j;
}

// Epilogues of the MFMA GEMM.
enum {
  EPI_BIAS = 0,      // out = C (+ bias)
  EPI_GELU_FWD = 1,  // out = C + bias (MLP pre-activation), out2 = GELU(out)
  EPI_GELU_BWD = 2,  // out = C * GELU'(aux)
  EPI_ITEM_QKV = 3,  // item Q|K|V + bias, written head-major; K, V for train rows only; K is
                     // stored times log2(e)/sqrt(d)
  EPI_LN = 4,        // out = LN(C + bias + resid); xhat, rstd saved
  EPI_LN_BWD = 5,    // dh = C + resid; out = LN'(dh) with xhat = aux, rstd_in; column partials
  EPI_DX = 6,        // out (native) = C (+ bias) + resid
  // pre-norm block
  EPI_RMS = 7,       // h = C + bias + rscale * resid -> out; out2 = gamma h rstd; rstd saved
  EPI_RMS_BWD = 8    // out (omode) = oscale (resid + RMS'(C)) with h = aux, rstd_in; column
                     // partials of C * h * rstd_in (the norm-weight gradient)
};

struct GemmArgs {
  int64_t M;
  int N, K, BN, epi;
  const bf16* A;
  const bf16* A2;  // ROWS_ITEM_HM: K and V arrays (A is Q)
  const bf16* A3;
  int64_t lda;
  int amode;
  const bf16* Bt;  // [N][K]
  const float* bias;
  bf16* out;
  bf16* out2;
  bf16* out3;
  int64_t ldo;
  int omode;
  const bf16* resid;
  int rmode;
  const float* gamma;
  const float* beta;
  bf16* xhat;
  float* rstd;
  const float* rstd_in;
  const bf16* aux;
  float* part;  // EPI_LN_BWD: [row tiles][2][BN] partial sums (dgamma, dbeta);
                //   EPI_RMS_BWD: [row tiles][BN] (dgamma)
  const float* rgamma;  // EPI_LN: resid read as rgamma * resid + rbeta per column (null: as is)
  const float* rbeta;
  int xhat_out;  // EPI_LN: out receives x-hat (the normalised rows) instead of gamma x-hat + beta
  float rscale;  // EPI_RMS: factor on resid
  float oscale;  // EPI_RMS_BWD: factor on the output
  float eps;     // EPI_RMS, EPI_RMS_BWD: RMSNorm epsilon
  Geo g;
};

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);

// Cells per block tile of the MFMA GEMM; EPI_LN_BWD writes one partial row per tile.
constexpr int GEMM_BM = 64;
inline int64_t gemm_row_tiles(int64_t M) { return (M + GEMM_BM - 1) / GEMM_BM; }
// Row tiles of one launch of epilogue epi at column tile BN (the launch picks 64 or 128 rows);
// never more than gemm_row_tiles(M).
int64_t gemm_tiles(int epi, int BN, int64_t M);

// bf16 copies of the six weight matrices of one layer, as stored ([out][in]) and transposed.
// Offsets (elements) inside w / wt follow the packed parameter order of the weights:
// Wqkv_f, Wo_f, Wqkv_i, Wo_i, W1, W2.
// bf16 weight copies (element offsets); fb: float32 folded biases (3E item Q|K|V, then H MLP
// up), at element fb of the bf16 buffer
// ms: the weight stream of the fused MLP forward (mlp_fwd_stream_elems elements)
struct WOff {
  int64_t qkv_f, o_f, qkv_i, o_i, w1, w2, fb, ms, total;
};
WOff weight_offsets(int E, int H);
// LayerNorm affines folded into the products that consume the normalised rows: the item Q|K|V
// projection reads x-hat1 with weights Wqkv_i diag(g1) and bias bqkv_i + Wqkv_i be1, the MLP
// up-projection x-hat2 with W1 diag(g2) and b1 + W1 be2 (null: no folding)
struct WFold {
  const float *g1, *be1, *bqkv_i, *g2, *be2, *b1;
};
// w: the six matrices in packed order (the fold applied to Wqkv_i and W1 when given, and the
// folded biases written at fb); wt: each matrix transposed, never folded
hipError_t launch_weight_prep(const float* params, int E, int H, bf16* w, bf16* wt,
                              const WFold* fold, hipStream_t s);

// Weight gradient of a product whose input was the folded x-hat (see WFold): with
// h = gamma o x-hat + beta, dW[n][k] = (sum_z wpart)[n][k] gamma[k] + (sum_z bpart)[n] beta[k];
// grad (N x K) = (accumulate ? grad : 0) + that, in the fixed summation order of
// launch_reduce_z.  The bias sums are left in the first row of bpart (the other rows are
// scratch afterwards): the bias gradient is then a one-row reduce of bpart.
hipError_t launch_reduce_wfold(int Z, int N, int K, float* wpart, float* bpart,
                               const float* gamma, const float* beta, float* grad,
                               int accumulate, hipStream_t s);

// Writes 0 to every element of the native tensor that lies in an inactive cell.
hipError_t launch_zero_inactive(const Geo& g, bf16* native, hipStream_t s);

// Weight gradient dW[n][k] = sum_m dY[m][n] X[m][k] (+ db[n] = sum_m dY[m][n]) over M cells,
// split into Z = wgrad_chunks(M) chunks of wgrad_chunk(M) cells (a multiple of 32, at most
// WGRAD_CHUNK_MAX): M / 256 cells rounded up while that is at most WGRAD_CHUNK_MAX, so that
// the workgroups of one tile fill the 256 compute units in whole rounds; partials land in part
// [Z][N][K] and bpart [Z][N].  wgrad_max_chunks(Mmax) bounds Z for every M <= Mmax.
constexpr int WGRAD_CHUNK_MAX = 8192;
constexpr int WGRAD_SLOTS = 256;
int64_t wgrad_chunk(int64_t M);
int64_t wgrad_max_chunks(int64_t Mmax);
struct WgradArgs {
  int64_t M;
  int N, K;
  const bf16* dY;  // compact rows, leading dimension ldy, or ROWS_ITEM_HM (dY, dY2, dY3)
  const bf16* dY2;
  const bf16* dY3;
  int64_t ldy;
  int ymode;
  const bf16* X;   // rows per xmode (compact with ldx, or the native cell tensor)
  int64_t ldx;
  int xmode;
  float* part;
  float* bpart;    // may be null: no bias gradient
  int64_t chunk;
  Geo g;
};
int wgrad_chunks(int64_t M);
hipError_t launch_wgrad_mfma(const WgradArgs& a, hipStream_t s);
// out[i] = (accumulate ? out[i] : 0) + sum_z part[z * stride + i], fixed summation order.
// With many partials and few outputs the sum runs in two passes, the first of which
// overwrites part (it is scratch).
hipError_t launch_reduce_z(int Z, int64_t count, int64_t stride, float* part, float* out,
                           int accumulate, hipStream_t s);

// Pre-norm block input: xs = decay * X (compact), r = gamma xs / sqrt(mean(xs^2) + eps)
// (compact), rstd [N].
hipError_t launch_rms_in(const Geo& g, const bf16* X, float decay, const float* gamma, float eps,
                         bf16* xs, bf16* r, float* rstd, hipStream_t s);

// Thinking rows: broadcast of table[T][E] into rows [0, T) of the native X (0 at inactive
// columns), and its gradient summed over datasets and active columns in a fixed order.
template <class TT>
hipError_t launch_thinking_fwd(const Geo& g, int T, const float* table, TT* X, hipStream_t s);
template <class TT>
hipError_t launch_thinking_bwd(const Geo& g, int T, const TT* dX, float* dtable, int accumulate,
                               hipStream_t s);

// Backward of the last LayerNorm from the native upstream gradient: dz = LN3'(dY) at active
// cells (compact), plus per-block partial column sums of dY * xhat and dY into
// part [blocks][2][E].  Returns the number of blocks through *nblocks.
hipError_t launch_ln_out_bwd(const Geo& g, const bf16* dY, const bf16* xhat, const float* rstd,
                             const float* gamma, bf16* dz, float* part, int* nblocks,
                             hipStream_t s);

// The MLP half of the post-norm block, forward, in one kernel (csrc/mlp.hip): item
// out-projection + residual + LN2, MLP up-projection, GELU and down-projection with the hidden
// layer in registers, residual + LN3.  Reads the weight stream that launch_mlp_fwd_stream
// builds (mlp_fwd_stream_elems(E, H) bf16 elements).
struct MlpFwdArgs {
  int64_t M;            // active cells
  const bf16* oi;       // [M][E] item attention output
  const bf16* xh1;      // [M][E] x-hat of LN1
  const bf16* ws;       // weight stream
  const float *bo, *g1, *be1, *g2, *be2, *b2, *g3, *be3;  // [E] each
  const float* fb1;     // [H] folded up-projection bias b1 + W1 be2
  bf16* xh2;            // [M][E] x-hat of LN2 (null: not stored)
  float* rs2;           // [M] (null: not stored)
  bf16* gout;           // [M][H] pre-activation (optional)
  bf16* uout;           // [M][H] GELU of it (optional)
  bf16* y;              // native [B][R][S][E]
  bf16* xh3;            // [M][E] x-hat of LN3 (null: not stored)
  float* rs3;           // [M] (null: not stored)
  Geo g;
};
bool mlp_fused_ok(int E, int H);
int64_t mlp_fwd_stream_elems(int E, int H);
hipError_t launch_mlp_fwd_stream(const float* wo, const float* w1, const float* g2,
                                 const float* w2, int E, int H, bf16* out, hipStream_t s);
hipError_t launch_mlp_fwd(const MlpFwdArgs& a, hipStream_t s);

// Backward of the same sub-block in one kernel (csrc/mlp.hip): LN3' from the native dY, the MLP
// backward with G recomputed from x-hat2, LN2'.  Writes dz3, dz2, dG and U (the weight
// gradients' operands) and per-tile column sums [mlp_bwd_tiles(M)][4 E]: dY xh3, dY, dh2 xh2,
// dh2 (the LN3 and LN2 weight and bias gradients).
struct MlpBwdArgs {
  int64_t M;
  const bf16* dy;       // native upstream gradient
  const bf16* xh3;      // [M][E]
  const float* rs3;     // [M]
  const bf16* xh2;      // [M][E]
  const float* rs2;     // [M]
  const bf16* ws;       // backward weight stream (mlp_bwd_stream_elems)
  const float *g3, *g2; // [E]
  const float* fb1;     // [H] folded up-projection bias
  bf16* dz3;            // [M][E]
  bf16* dz2;            // [M][E]
  bf16* dg;             // [M][H]
  bf16* u;              // [M][H]
  float* part;          // [mlp_bwd_tiles(M)][4 E]
  Geo g;
};
int64_t mlp_bwd_stream_elems(int E, int H);
int64_t mlp_bwd_tiles(int64_t M);
hipError_t launch_mlp_bwd_stream(const float* w1, const float* g2, const float* w2, int E, int H,
                                 bf16* out, hipStream_t s);
hipError_t launch_mlp_bwd(const MlpBwdArgs& a, hipStream_t s);

// Bytes of the LayerNorm-backward column partials for up to `cells` cells.
size_t ln_partial_bytes(int64_t cells, int E);

// Scratch bytes that the MFMA path needs inside the workspace.
size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16);

}  // namespace tfm
