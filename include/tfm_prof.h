/*
 * tfm_prof.h — optional per-step timing of the library's kernel launches.
 *
 * For measurement tools (the benchmark): while profiling is on, every launch step of
 * tfm_layer_fwd / tfm_layer_bwd is bracketed by two HIP events recorded on the caller's
 * stream, and the elapsed times are summed per step name.  Profiling adds two event records
 * per step and nothing else; it is off by default.  Not thread-safe: profile from one thread.
 */
#ifndef TFM_PROF_H
#define TFM_PROF_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Clears earlier records and turns event recording on (on != 0) or off.  Returns 0, or
 * TFM_ERR_HIP (-6) if the events cannot be created. */
int tfm_prof_enable(int on);

/* Waits for the recorded events and aggregates them.  Returns the number of distinct steps
 * recorded since tfm_prof_enable(1), or a negative code. */
int tfm_prof_collect(void);

/* Step i of the last tfm_prof_collect(): name (static string), number of launches and their
 * summed duration in milliseconds.  Returns 0, or -1 if i is out of range. */
int tfm_prof_step(int i, const char** name, long long* launches, double* total_ms);

/* Attribution of the item-attention backward to steps, for tools that price each step: on the
 * bfloat16 MFMA path the columns whose train prefix has at most this many rows run in the
 * one-kernel backward (step "item_attn_bwd"); longer prefixes run in the two-kernel form
 * (steps "item_attn_dq" and "item_attn_dkdv").  Returns 0 when head_dim has no one-kernel form.
 * Pure host function: no device, no side effects. */
int tfm_prof_item_bwd_fused_rows(int head_dim);

#ifdef __cplusplus
}
#endif

#endif /* TFM_PROF_H */
