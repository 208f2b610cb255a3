// Kernels of the two ends of the stack: the feature and target encoders that build the stack
// input, and the decoder with the cross-entropy loss that reads the stack output (paper, Fig. 3
// and Fig. 4 captions; App. "Repeated Feature Grouping" and "Autoresearch").
#pragma once

#include "common.h"

namespace tfm {

constexpr int ENDS_GMAX = 8;    // largest feature group
constexpr int ENDS_KMAX = 64;   // most decoder outputs
constexpr int ENC_ROWS = 16;    // data rows per encoder workgroup

// Per-dataset metadata on the device.
struct EndsDs {
  int32_t n_train;  // train rows of the stack input, thinking rows included
  int32_t n_feat;   // feature columns m = feature cells [0, m)
  int32_t n_class;  // classes: logits [0, n_class) enter the softmax
  int32_t test0;    // first decoder row of the dataset (test rows of earlier datasets)
};

struct EndsGeo {
  int32_t B, R, S, E;     // stack input [B][R][S][E], S = C + 1 (cell C is the target)
  int32_t T;              // thinking rows: data row i is row T + i of the stack input
  int32_t F;              // columns of a row of the feature array
  int32_t G;              // feature group size
  int32_t off[ENDS_GMAX]; // group shifts
  int32_t Hd, K;          // decoder hidden width and outputs
  int32_t mean;           // decoder input: 0 target cell, 1 mean of the feature cells
  int64_t Ttot;           // decoder rows = test rows of the whole batch
  const EndsDs* ds;       // [B]
};

// Encoder output rows [T, R) of every dataset: feature cells, zero padding cells, target cell.
template <class T>
hipError_t launch_encode_fwd(const EndsGeo& g, const float* x, const int32_t* lab,
                             const float* prm, T* X, hipStream_t s);
// Number of partial rows launch_encode_bwd writes (E * (G + 3) floats each).
int64_t encode_bwd_parts(const EndsGeo& g);
template <class T>
hipError_t launch_encode_bwd(const EndsGeo& g, const float* x, const int32_t* lab, const T* dX,
                             float* part, hipStream_t s);

// Decoder input Z[Ttot][E] (float32) from the stack output Y.
template <class T>
hipError_t launch_decode_gather(const EndsGeo& g, const T* Y, float* Z, hipStream_t s);
// dY over the whole stack output: the decoder input's gradient at the decoded cells of the test
// rows (divided by m for the mean), 0 elsewhere.
template <class T>
hipError_t launch_decode_scatter(const EndsGeo& g, const float* dZ, T* dY, hipStream_t s);
// Masked softmax cross entropy per decoder row: lrow[t] = loss / Ttot, dlog = gradient of the
// batch mean (0 for classes past the dataset's count).
hipError_t launch_cross_entropy(const EndsGeo& g, const float* logits, const int32_t* lab,
                                float* lrow, float* dlog, hipStream_t s);

// float32 GEMM on the fp32 MFMA: C[M][N] = op(A)[M][K] op(B)[K][N] with an epilogue.
// op(A)[m][k] = TA ? A[k*lda + m] : A[m*lda + k]; op(B)[k][n] = TB ? B[n*ldb + k] : B[k*ldb + n].
enum { SG_BIAS = 0, SG_GELU = 1, SG_GELU_GRAD = 2, SG_AXPBY = 3 };
struct SgemmArgs {
  const float* A;
  const float* B;
  float* C;
  float* C2;          // SG_GELU: GELU(C)
  const float* bias;  // [N] or null (SG_BIAS, SG_GELU)
  const float* aux;   // SG_GELU_GRAD: pre-activation, C = acc * GELU'(aux);
                      // SG_AXPBY: C = alpha * acc + beta * aux  ([M][ldc] like C)
  float alpha, beta;
  int64_t lda, ldb, ldc;
  int32_t M, N, K;
  int32_t kchunk;     // split-K: grid.z chunks of kchunk (multiple of 16); 0 = whole K
  int64_t zstride;    // offset of grid.z index z's output (split-K partials, or batch entries)
  int32_t batch;      // kchunk == 0: grid.z runs over `batch` independent products whose A,
  int64_t bsa, bsb;   // B and aux lie bsa, bsb and bsaux floats apart (C zstride apart)
  int64_t bsaux;
};
hipError_t launch_sgemm(const SgemmArgs& a, bool ta, bool tb, int epi, hipStream_t s);

// p[i] = v for i in [0, n) (a kernel, so that the call can sit in a captured graph).
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s);

// Shared with the C-ABI source of the layer: set the thread's last error (returns code), and
// validate a tfm_dims as every layer entry point does (0 or a negative code).
int abi_fail(int code, const char* msg);
int abi_check_dims(const void* dims);

}  // namespace tfm
