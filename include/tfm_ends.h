/*
 * tfm_ends.h — C ABI of the two ends of the stack on MI355X (gfx950): the encoders that turn a
 * batch of tables into the stack input, and the decoder with the cross-entropy loss that turns
 * the stack output into the training loss (paper "Speedrunning Tabular Foundation Model
 * Pretraining", Fig. 3 and Fig. 4 captions, Tab. 5, App. "Repeated Feature Grouping" and
 * "Autoresearch").  With tfm_layer.h this covers a whole training step:
 *
 *     X  = encode(x, labels)             tfm_encode_fwd   (+ tfm_thinking_rows_fwd)
 *     Y  = blocks(X)                     tfm_layer_fwd per block
 *     loss, dY, decoder grads            tfm_decode_loss
 *     dX, block grads                    tfm_layer_bwd per block
 *     encoder grads                      tfm_encode_bwd   (+ tfm_thinking_rows_bwd)
 *
 * Encoders.  A table b has m = n_feat[b] feature columns.  Feature cell j in [0, m) of a row holds
 *     W_fe [x_{(j+o_0) mod m}, ..., x_{(j+o_{G-1}) mod m}] + b_fe
 * (one group per column, led by column j; G = 1, o_0 = 0 encodes each feature alone), cells
 * [m, C) are padding (written as 0) and the target cell C holds t W_te + b_te, where t is the
 * row's class index for a labelled row and, for an unlabelled row, the mean class index of the
 * labelled rows — so no unlabelled row's label reaches the stack.  The stack's cell_mask for
 * such a batch is cells [0, m) plus the target cell.
 *
 * Decoder.  For every unlabelled row, in (dataset, row) order, z is the target cell of the stack
 * output (decode_mean == 0, the baseline) or the mean of its m feature cells (decode_mean == 1,
 * the current best record); logits = W_d2 GELU(W_d1 z + b_d1) + b_d2 with exact-erf GELU.  A
 * dataset with k = n_class[b] classes takes the softmax over logits [0, k); the loss is the
 * cross entropy of the rows' labels, averaged over every unlabelled row of the batch.
 *
 * Conventions (as tfm_layer.h unless stated):
 *   - dims: the stack's tfm_dims (B, R, C, E, dtype); heads, H and block are not used here but
 *     must be valid.  The stack input/output X, Y, dY, dX: device [B][R][C+1][E], dims->dtype.
 *   - Thinking rows: rows [0, T) of the stack input are thinking rows (ends->T, written by
 *     tfm_thinking_rows_fwd); data row i is stack row T + i.  n_train counts thinking rows, so
 *     data rows [0, n_train[b] - T) are labelled; n_train[b] must lie in [T + 1, R].
 *   - x: device float32 [B][R - T][F], row i of table b at x + (b (R - T) + i) F; columns
 *     [0, n_feat[b]) are read.  labels: device int32 [B][R - T] class indices; the encoders read
 *     the labelled rows' entries, the decoder the unlabelled rows' entries, which must lie in
 *     [0, n_class[b]) (another value gives that row an undefined loss, never an out-of-bounds
 *     access).
 *   - n_train, n_feat, n_class: host int32[B]; n_feat[b] in [1, min(C, F)], n_class[b] in [1, K].
 *   - params, grads: device float32, one packed vector of tfm_ends_param_count() floats:
 *         W_fe[E][G] b_fe[E] W_te[E] b_te[E]          encoders
 *         W_d1[Hd][E] b_d1[Hd] W_d2[K][Hd] b_d2[K]     decoder
 *     tfm_encode_bwd writes the encoder entries of grads, tfm_decode_loss the decoder entries;
 *     neither touches the other's.  accumulate != 0 adds to grads instead of overwriting.
 *   - workspace: device scratch of tfm_ends_workspace_bytes(); contents are not preserved.
 *   - Parameter gradients and the loss are reduced in a fixed order (bitwise reproducible).
 *   - All device pointers must be non-null and 16-byte aligned; the caller owns every buffer,
 *     the library allocates nothing; calls are asynchronous on `stream`; on a negative return
 *     nothing was launched and tfm_last_error() describes the error.
 */
#ifndef TFM_ENDS_H
#define TFM_ENDS_H

#include "tfm_layer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Shape of the ends. */
typedef struct {
  int32_t G;           /* feature group size, 1..8 */
  int32_t offsets[8];  /* group shifts offsets[0..G-1], each in [0, 2^20] */
  int32_t F;           /* columns per row of x, >= 1 */
  int32_t T;           /* thinking rows at the head of the stack input, 0 <= T < R */
  int32_t Hd;          /* decoder hidden width, 1..4096 */
  int32_t K;           /* decoder outputs, 1..64 */
  int32_t decode_mean; /* 0: decode the target cell; 1: the mean of the feature cells */
} tfm_ends;

/* Float32 parameters of the ends: E G + 3 E + Hd E + Hd + K Hd + K (0 on invalid arguments). */
size_t tfm_ends_param_count(const tfm_dims* dims, const tfm_ends* ends);

/* Bytes of scratch of any ends call with these dims (0 on invalid arguments). */
size_t tfm_ends_workspace_bytes(const tfm_dims* dims, const tfm_ends* ends);

/* Encoder forward (Fig. 3; App. "Repeated Feature Grouping"): writes rows [T, R) of every cell
 * of X; rows [0, T) are left untouched. */
int tfm_encode_fwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const float* x, const int32_t* labels,
                   const float* params, void* X, void* workspace, size_t workspace_bytes,
                   void* stream);

/* Encoder gradients for the gradient dX of the stack input (rows [T, R); padding cells are
 * ignored). */
int tfm_encode_bwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const float* x, const int32_t* labels, const void* dX,
                   float* grads, int accumulate, void* workspace, size_t workspace_bytes,
                   void* stream);

/* Decoder forward only (evaluation): logits, device float32 [T_test][K] with T_test the number
 * of unlabelled rows of the batch, in (dataset, row) order; entries past a dataset's class
 * count are written as computed (the caller ignores them).  Here n_train[b] may be anything in
 * [0, R] (T is not used): rows [n_train[b], R) are decoded, so the stack output of a chunk of
 * unlabelled rows from the forward-only query calls of tfm_layer.h (n_train = 0) can be
 * decoded directly. */
int tfm_decode_fwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const void* Y, const float* params, float* logits,
                   void* workspace, size_t workspace_bytes, void* stream);

/* Decoder and loss, forward and backward (Fig. 3 and 4 captions; App. "Autoresearch"):
 * loss (device float32 [1]) = mean cross entropy over the unlabelled rows (0 if there are none);
 * logits (nullable) as tfm_decode_fwd; dY (whole stack output, dims->dtype) = the loss's
 * gradient, zero except at the decoded cells of unlabelled rows; the decoder entries of grads. */
int tfm_decode_loss(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                    const int32_t* n_feat, const int32_t* n_class, const int32_t* labels,
                    const void* Y, const float* params, float* loss, float* logits, void* dY,
                    float* grads, int accumulate, void* workspace, size_t workspace_bytes,
                    void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TFM_ENDS_H */
