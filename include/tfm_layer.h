/*
 * tfm_layer.h — C ABI of the MI355X (gfx950) two-axis tabular transformer layer.
 *
 * The layer (paper "Speedrunning Tabular Foundation Model Pretraining", Sec. 4.1 and the
 * Fig. 3 caption; Tab. 5 for the baseline sizes) maps a cell tensor X[B, R, C+1, E] — B
 * datasets (tables), R rows each, C feature cells plus one target cell per row, embedding
 * width E — to Y of the same shape:
 *
 *     H1 = LN1(X  + FeatureAttention(X))    attention across the active cells of each row
 *     H2 = LN2(H1 + ItemAttention(H1))      attention down each column; every row attends only
 *                                           to the first n_train[b] (labelled) rows
 *     Y  = LN3(H2 + W2 GELU(W1 H2 + b1) + b2)
 *
 * Post-norm LayerNorms (eps 1e-5, biased variance, affine), exact-erf GELU, attention scale
 * 1/sqrt(E/heads), two independent attention parameter sets, bias on every linear.
 *
 * Memory conventions
 *   - X, Y, dY, dX: device, row-major [B][R][C+1][E], element type per dims->dtype
 *     (TFM_F32: float, TFM_BF16: bfloat16 bit patterns).
 *   - params, grads: device, float32, one packed vector per layer of
 *     tfm_layer_param_count() floats, in this order (weights row-major [out][in]):
 *         Wqkv_f[3E][E] bqkv_f[3E] Wo_f[E][E] bo_f[E]       feature-axis attention
 *         Wqkv_i[3E][E] bqkv_i[3E] Wo_i[E][E] bo_i[E]       item-axis attention
 *         W1[H][E] b1[H] W2[E][H] b2[E]                     MLP
 *         g1[E] be1[E] g2[E] be2[E] g3[E] be3[E]            LayerNorm scales and shifts
 *     Rows [0,E) of Wqkv are Q, [E,2E) K, [2E,3E) V; head j owns rows [j*d, (j+1)*d) of each.
 *   - n_train: host int32[B], each in [1, R]; rows [0, n_train[b]) of dataset b are its
 *     train (labelled) rows and the only keys of the item-axis attention.
 *   - cell_mask: host uint8[B][C+1]; non-zero = active cell column.  The target cell (index
 *     C) must be active.  Inactive cells are inert: never keys or queries, Y and dX are
 *     written as 0 there, dY there is ignored, and they add nothing to any gradient.
 *   - saved: device buffer of tfm_layer_saved_bytes(), written by fwd, read by bwd.
 *   - workspace: device scratch of tfm_layer_workspace_bytes(); contents are not preserved.
 *   - stream: a hipStream_t (passed as void*); NULL means the null stream.
 *
 * All pointers must be 16-byte aligned.  The caller owns every buffer; the library allocates
 * no device memory and keeps no state between calls.  Calls are asynchronous on `stream`
 * and never synchronise the device.  Every entry point validates its arguments before it
 * launches anything: on error nothing is launched, the return code is negative and
 * tfm_last_error() describes it.
 *
 * Supported envelope: B >= 1, R >= 1, 0 <= C <= 255, heads >= 1, d = E/heads in {16, 32, 64},
 * 32 <= E <= 256 with E % 32 == 0, 32 <= H <= 1024 with H % 32 == 0, at most 2^26 cells
 * B*R*(C+1) in all, and R*(C+1)*E <= 715,827,882 (one dataset's bfloat16 Q|K|V under 4 GiB).
 *
 * Pre-norm block (dims->block == TFM_BLOCK_PRENORM): the block of the paper's current best
 * record (Sec. 5 "Residual Decay" and "RMSNorm, Thinking Rows", the Fig. 4 caption, App. B.6,
 * Tab. 5), with c = dims->decay (0.95^i for block i of a stack):
 *
 *     X' = c X
 *     H1 = X' + FeatureAttention(RMS1(X'))
 *     H2 = H1 + ItemAttention(RMS2(H1))
 *     Y  = H2 + W2 GELU(W1 RMS3(H2) + b1) + b2,      RMS(u) = g * u / sqrt(mean(u^2) + 1e-6)
 *
 * Its packed parameters are those of the post-norm block without the shifts, ending
 * g1[E] g2[E] g3[E] (RMSNorm weights).  Thinking rows are train rows that the caller prepends
 * (n_train counts them); inside the block they are ordinary rows.  The pre-norm block runs in
 * bfloat16 only, with E in {64, 128, 192, 256} and H a multiple of E.
 */
#ifndef TFM_LAYER_H
#define TFM_LAYER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { TFM_F32 = 0, TFM_BF16 = 1 } tfm_dtype;
typedef enum { TFM_BLOCK_POSTNORM = 0, TFM_BLOCK_PRENORM = 1 } tfm_block;

/* Problem dimensions.  C counts feature cells; each row has S = C + 1 cells.  block selects
 * the layer variant (a zero-initialised struct selects the post-norm block); decay is the
 * factor the pre-norm block multiplies its input by (ignored by the post-norm block). */
typedef struct {
  int32_t B, R, C, E, heads, H;
  int32_t dtype; /* tfm_dtype */
  int32_t block; /* tfm_block */
  float decay;
} tfm_dims;

/* Return codes. */
enum {
  TFM_OK = 0,
  TFM_ERR_DIMS = -1,      /* dimension outside the supported envelope */
  TFM_ERR_HEAD_DIM = -2,  /* E % heads != 0 or d = E/heads not in {16, 32, 64} */
  TFM_ERR_NTRAIN = -3,    /* some n_train[b] outside [1, R] (query calls: [1, context_rows]) */
  TFM_ERR_MASK = -4,      /* target cell of some dataset inactive */
  TFM_ERR_POINTER = -5,   /* null or misaligned pointer */
  TFM_ERR_HIP = -6,       /* a HIP launch failed */
  TFM_ERR_BUFFER = -7     /* saved, workspace or cache buffer smaller than required */
};

/* Number of float32 parameters of one layer: 8E^2 + 8E + 2EH + H + 7E. 0 on invalid dims. */
size_t tfm_layer_param_count(const tfm_dims* dims);

/* Bytes of the fwd->bwd state buffer; depends on dims only (sized for all cells active). */
size_t tfm_layer_saved_bytes(const tfm_dims* dims);

/* Bytes of scratch that fwd and bwd need; depends on dims only. */
size_t tfm_layer_workspace_bytes(const tfm_dims* dims);

/* Forward pass (Sec. 4.1 / Fig. 3 block).  Reads X and params, writes Y and saved. */
int tfm_layer_fwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                  const void* X, const float* params, void* Y,
                  void* saved, size_t saved_bytes, void* workspace, size_t workspace_bytes,
                  void* stream);

/* Backward pass of the same layer.  X, params, n_train and cell_mask must equal those of the
 * forward call that wrote `saved`.  Writes dX; writes grads (accumulate == 0) or adds to them
 * (accumulate != 0).  Parameter gradients are sums over every active cell of every dataset,
 * reduced in a fixed order (bitwise reproducible). */
int tfm_layer_bwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                  const void* X, const float* params, const void* saved, size_t saved_bytes,
                  const void* dY, void* dX, float* grads, int accumulate,
                  void* workspace, size_t workspace_bytes, void* stream);

/* Allocation-free forward, for callers that cannot allocate device memory or pass a workspace
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments and results as tfm_layer_fwd (Y and saved bit for bit; saved feeds tfm_layer_bwd as
 * usual) without the workspace: the call's scratch (the active-cell plan and the bfloat16 copies
 * of the weights) lives in a device array the library owns, TFM_NOALLOC_SCRATCH_BYTES on each
 * GPU it runs on, held until the process ends.  The call allocates nothing and calls no
 * allocating routine.
 *
 * Limits: TFM_BF16 with E in {64, 128, 192, 256} and H a multiple of E (either block); dims whose
 * scratch exceeds TFM_NOALLOC_SCRATCH_BYTES (the bf16 weights, 2 (8E^2 + 2EH) bytes, plus about
 * 24 B (C+1) + 28 + 4 ceil((C+1)/32) bytes per dataset) return TFM_ERR_BUFFER; a stream of another
 * device than the current one returns TFM_ERR_HIP.  The array is shared by every call on one
 * GPU and keeps the last call's contents (nothing in it needs to start at zero: each call
 * rewrites what it reads), so calls that overlap on one GPU (concurrent streams, or threads)
 * race: the caller serialises them. */
#define TFM_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int tfm_layer_fwd_noalloc(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          const void* X, const float* params, void* Y, void* saved,
                          size_t saved_bytes, void* stream);

/* Thinking rows (Sec. 5 "RMSNorm, Thinking Rows", App. B.6, Tab. 5): learned E-vectors
 * prepended along the row axis, broadcast over the cell columns and counted as train rows.
 * dims, n_train and cell_mask describe the stack input X[B][R][C+1][E] whose rows [0, T) are the
 * thinking rows (n_train includes them, 1 <= T <= min(n_train)); workspace is a
 * tfm_layer_workspace_bytes() or tfm_infer_workspace_bytes() scratch (only its leading bytes
 * are used: the column map).
 *
 * tfm_thinking_rows_fwd writes table[T][E] (device, float32, rounded to dims->dtype) into rows
 * [0, T) of every active cell column of X and 0 into rows [0, T) of inactive columns; other rows
 * are left untouched. */
int tfm_thinking_rows_fwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          int T, const float* table, void* X, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Gradient of the broadcast: dtable[T][E] (device, float32) = sum over datasets and active cell
 * columns of dX rows [0, T), added to dtable when accumulate != 0, summed in a fixed order. */
int tfm_thinking_rows_bwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          int T, const void* dX, float* dtable, int accumulate, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Forward-only (inference) calls: the evaluation of Sec. 3 "Evaluation" and App. "Evaluation
 * Pipeline" runs the model forward on the train folds of a table as labelled rows and on the
 * held-out fold as unlabelled ones, in bf16 autocast (the inference row of the ablation table of
 * App. "SDPA, bf16, LR, Width").  No row attends to an unlabelled row, so the keys and values
 * of the item-axis attention depend on the train rows only.  The calls exploit that:
 *
 *   tfm_layer_fwd_context  runs the layer forward on X[B][R][C+1][E] exactly as tfm_layer_fwd
 *       does (same Y, bit for bit), keeps nothing for a backward pass, and writes the item-axis
 *       keys and values of the train rows [0, n_train[b]) into kv_cache.
 *   tfm_layer_fwd_query    runs the layer forward on further rows Xq[B][Rq][C+1][E] (dims->R =
 *       Rq) that are all unlabelled: each attends, on the item axis, to the n_train[b] keys and
 *       values a context call left in kv_cache.  Its Y equals the rows a tfm_layer_fwd call on
 *       [context rows; query rows] would give them.
 *
 * So a stack of layers encodes the train rows once (a context call per layer, one cache per
 * layer) and then answers any number of query chunks, each through all layers, with memory
 * proportional to the chunk.  Both calls need TFM_BF16 and E in {64, 128, 192, 256} with H a
 * multiple of E (either block).  The query call needs the n_train, cell_mask, params and dims
 * (other than R) of the context call that wrote kv_cache, and context_rows = that call's R;
 * n_train[b] must lie in [1, context_rows]. */

/* Bytes of scratch of one forward-only call with dims->R rows (0 on invalid or unsupported
 * dims). */
size_t tfm_infer_workspace_bytes(const tfm_dims* dims);

/* Bytes of the key/value cache of one layer whose context call has dims->R rows (opaque
 * layout: keys and values of every possible active column, head-major, bfloat16). */
size_t tfm_infer_cache_bytes(const tfm_dims* dims);

int tfm_layer_fwd_context(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          const void* X, const float* params, void* Y, void* kv_cache,
                          size_t cache_bytes, void* workspace, size_t workspace_bytes,
                          void* stream);

int tfm_layer_fwd_query(const tfm_dims* dims, int32_t context_rows, const int32_t* n_train,
                        const uint8_t* cell_mask, const void* X, const float* params,
                        const void* kv_cache, size_t cache_bytes, void* Y, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Message describing the last non-zero return of this thread ("" if none). */
const char* tfm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TFM_LAYER_H */
