/*
 * tfm_optim.h — C ABI of the optimiser step on MI355X (gfx950) (paper "Speedrunning Tabular
 * Foundation Model Pretraining", Sec. 5 "Muon Optimizer" and "Batched Muon, Compile", App.
 * "Muon Optimizer", "Batched Muon, Compile", "LAWA, AdamW Weight Decay", Tab. 5): clipping of the
 * gradients by their global norm, Muon on the hidden weight matrices of the blocks with the
 * Newton–Schulz iteration batched over equally shaped matrices (the Q, K and V matrices of a
 * block, and the same matrices of every block), and schedule-free AdamW on the other parameters.
 *
 * Conventions: every array is device float32 unless stated; the caller owns every buffer and the
 * library allocates nothing; calls are asynchronous on `stream` (a hipStream_t, NULL = the null
 * stream); device pointers must be non-null and 16-byte aligned (matrices and vectors handed
 * over as lists may start anywhere on a 4-byte boundary); results are reduced in a fixed order
 * (bitwise reproducible); on a negative return (the codes of tfm_layer.h) nothing was launched
 * and tfm_last_error() describes the error.
 */
#ifndef TFM_OPTIM_H
#define TFM_OPTIM_H

#include "tfm_layer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ---- gradient clipping (Tab. 5 "Gradient clip") --------------------------------------------
 * norm = the L2 norm of the concatenation of nvec gradient arrays grads[i] (counts[i] floats
 * each; host arrays of device pointers and counts, nvec in [1, 1024]); scale = min(1, max_norm /
 * (norm + 1e-6)), the factor the optimisers below take as grad_scale.  scale and norm (nullable)
 * are device float32 [1]. */
size_t tfm_clip_workspace_bytes(int32_t nvec, const int64_t* counts);
int tfm_clip_scale(int32_t nvec, const float* const* grads, const int64_t* counts, float max_norm,
                   float* scale, float* norm, void* workspace, size_t workspace_bytes,
                   void* stream);

/* ---- schedule-free AdamW (App. "Baseline": the baseline's optimiser; Tab. 5) ----------------
 * One step t >= 1 of schedule-free AdamW (Defazio et al. 2024, AdamW form) on the entries of the
 * nseg segments [seg_off[k], seg_off[k] + seg_len[k]) (host int64 arrays, nseg in [1, 64],
 * segments disjoint) of the vectors y (the model's parameters, where the gradient was taken),
 * z (the base sequence, equal to y before the first step) and v (second moments, 0 before the
 * first step).  With g = grad_scale[0] * grad (grad_scale nullable = 1), s_t = lr min(1, t /
 * warmup) (1 without warm-up), gamma_t = s_t sqrt(1 - beta2^t) and the averaging weight
 * c = gamma_t^2 / sum_{i<=t} gamma_i^2 (Defazio et al.'s Algorithm 1):
 *     v <- beta2 v + (1 - beta2) g^2,   u = g / (sqrt(v) + eps) + weight_decay y,
 *     y <- y + c (z - y) + gamma_t (beta1 (1 - c) - 1) u,   z <- z - gamma_t u.
 * Entries outside the segments are not touched. */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
  int32_t warmup; /* steps of linear warm-up, 0 = none */
} tfm_sfadamw;

int tfm_sfadamw_step(const tfm_sfadamw* hp, int64_t t, int32_t nseg, const int64_t* seg_off,
                     const int64_t* seg_len, float* y, float* z, float* v, const float* grad,
                     const float* grad_scale, void* stream);

/* ---- Muon (Sec. 5 "Muon Optimizer", "Batched Muon, Compile") ---------------------------------
 * One Muon step on `count` matrices of the same shape rows x cols (row-major, W[i], G[i] and
 * buf[i] given as host arrays of device pointers; count in [1, 1024], rows and cols in
 * [1, 8192]).  With g = grad_scale[0] * G[i] (grad_scale nullable = 1):
 *     buf <- momentum buf + (1 - momentum) g,   U = nesterov ? (1 - momentum) g + momentum buf
 *                                                            : buf,
 *     O = ns_steps quintic Newton–Schulz steps X <- a X + b (X X^T) X + c (X X^T)^2 X,
 *         (a, b, c) = (3.4445, -4.7750, 2.0315), on U^T if rows > cols else U, scaled to unit
 *         Frobenius norm (guard 1e-7) first, transposed back,
 *     W <- W (1 - lr weight_decay) - lr max(1, rows / cols)^(1/2) O.
 * The iteration runs in float32 on the matrix cores, batched over the count matrices. */
typedef struct {
  float lr, momentum, weight_decay;
  int32_t nesterov; /* non-zero: Nesterov look-ahead */
  int32_t ns_steps; /* Newton–Schulz steps, 1..16 (5 in the published method) */
} tfm_muon;

size_t tfm_muon_workspace_bytes(int32_t count, int32_t rows, int32_t cols);
int tfm_muon_step(const tfm_muon* hp, int32_t count, int32_t rows, int32_t cols, float* const* W,
                  const float* const* G, float* const* buf, const float* grad_scale,
                  void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TFM_OPTIM_H */
