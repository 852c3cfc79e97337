/*
 * mar_kernels.h - per-kernel entry points of the cached MAR step.
 *
 * The same kernels mar_step runs, exposed one at a time so that each step of
 * the path can be checked on its own.  Conventions as in mar_cache.h:
 * device pointers, row-major dense layouts, `dtype` is mar_dtype (storage
 * type; products accumulate in fp32), asynchronous on `stream`, arguments
 * checked on the host before any launch (an error launches nothing).
 * Buffers read or written in 16-byte vectors must be 16-byte aligned.
 *
 * Row mapping used below: with `idx` given, row m of a compact matrix belongs
 * to slot m / per_slot and token idx[m] of that slot; without it, row m is
 * token m % per_slot of slot m / per_slot (and per_slot must equal seq).
 * The key and value caches [slots, H, seq, d_head] hold one slot's keys (or
 * values) of head h as a contiguous seq x d_head block.
 */
#ifndef MAR_KERNELS_H
#define MAR_KERNELS_H

#include <stdint.h>

#include "mar_cache.h"

#ifdef __cplusplus
extern "C" {
#endif

/* LayerNorm of the pre-LN block (LN1 / LN2), optionally gathering the rows
 * first (Eq. 9: only the computed rows enter blocks P..L-1).
 *   out[m]      = (r - mean(r)) / sqrt(var(r) + eps) * w + b   in dtype
 *   copy_f32[m] = r (nullable)
 * with r the source row of m: src is [slots, seq, d] (fp32 if src_f32 else
 * dtype), m < `m`.  Statistics in fp32, biased variance.  d % 8 == 0,
 * d <= 2048; src, w, b, out and copy_f32 16-byte aligned (MAR_E_ARG
 * otherwise). */
mar_status mar_k_layernorm(int32_t dtype, const void* src, int32_t src_f32, const int32_t* idx,
                           int32_t per_slot, int32_t seq, int32_t m, int32_t d, const float* w,
                           const float* b, float eps, float* copy_f32, void* out, void* stream);

/* out[m, n] = act(a w^T + bias) in dtype; a [m, k], w [n, k] (nn.Linear
 * layout), bias [n] fp32; act = exact-erf GELU when `act` != 0 (the block's
 * first MLP product), identity otherwise.  k % 64 == 0, n % 8 == 0; a, w
 * and out 16-byte aligned (MAR_E_ARG otherwise). */
mar_status mar_k_linear(int32_t dtype, int32_t act, const void* a, const void* w, const float* bias,
                        int32_t m, int32_t n, int32_t k, void* out, void* stream);

/* Residual product (output projection, second MLP product):
 *   x[m, n] = resid[m, n] + (a w^T)[m, n] + bias[n]      fp32
 * written to out[m, n] (out may equal resid), or, when out_idx is given, to
 * out[(m / per_slot) * seq + out_idx[m], n] (the scatter of the fresh rows
 * into the output cache, Eq. 9) with resid_copy[m, n] = x (nullable).
 * k % 64 == 0, n % 8 == 0; a, w, resid, out and resid_copy 16-byte
 * aligned (MAR_E_ARG otherwise). */
mar_status mar_k_linear_residual(int32_t dtype, const void* a, const void* w, const float* bias,
                                 int32_t m, int32_t n, int32_t k, const float* resid, float* out,
                                 const int32_t* out_idx, int32_t per_slot, int32_t seq,
                                 float* resid_copy, void* stream);

/* Query/key/value projection with the key/value cache update (Eq. 9: the
 * computed rows replace their cached keys and values).  Columns
 * [n_offset, n_offset + n_cols) of the stacked [3D, D] projection, with w
 * and bias pointing at column n_offset:
 *   query columns  -> q_out[m, c]                  ([m, D], dtype)
 *   key columns    -> k_cache[slot, head, tok, :]  ([slots, H, seq, dh])
 *   value columns  -> v_cache[slot, head, tok, :]  ([slots, H, seq, dh];
 *                     nullable) and v_copy, a second buffer of the same
 *                     layout (nullable); one of them required
 * slot/tok from the row mapping.  d_model % 64 == 0, d_head % 16 == 0,
 * n_offset % 32 == 0, n_cols % 8 == 0; every matrix argument 16-byte
 * aligned (MAR_E_ARG otherwise). */
mar_status mar_k_qkv(int32_t dtype, const void* a, const void* w, const float* bias, int32_t m,
                     int32_t n_cols, int32_t n_offset, int32_t d_model, int32_t n_heads, int32_t seq,
                     int32_t per_slot, const int32_t* idx, void* q_out, void* k_cache, void* v_cache,
                     void* v_copy, void* stream);

/* Eq. (3) without mask for per_slot query rows per slot against all seq
 * keys of the slot: q, out [n_slots * per_slot, H * d_head] (head h at
 * columns h * d_head ...), k and v [n_slots, H, seq, d_head] (the cache
 * layout).  Scale
 * 1/sqrt(d_head); softmax statistics in fp32.  d_head in {16, 32, ..., 128}.
 * per_slot == seq is the dense block; per_slot = N the cached one.  q, k,
 * v and out 16-byte aligned (MAR_E_ARG otherwise). */
mar_status mar_k_attention(int32_t dtype, const void* q, const void* k, const void* v, void* out,
                           int32_t n_slots, int32_t n_heads, int32_t seq, int32_t d_head,
                           int32_t per_slot, void* stream);

/* Eq. (8) similarity of every token: scores[slot, t] (fp64) = cosine of
 * v_cur and v_ref rows (layout [n_slots, H, seq, d_head]; a token's row is
 * its d_head slices over all heads), products and sums in fp64; 1 if both
 * rows are zero, 0 if one is.  With update_ref != 0, v_ref receives v_cur
 * afterwards.  d_head % 8 == 0; v_cur and v_ref 16-byte aligned
 * (MAR_E_ARG otherwise). */
mar_status mar_k_scores(int32_t dtype, const void* v_cur, void* v_ref, int32_t n_slots, int32_t n_heads,
                        int32_t seq, int32_t d_head, double* scores, int32_t update_ref, void* stream);

/* Eq. (8) selection: idx[slot, 0..n) = the n tokens of the slot with the
 * smallest score (NaN ranks as +inf, ties to the lower index), ascending.
 * seq <= 4096. */
mar_status mar_k_select(const double* scores, int32_t n_slots, int32_t seq, int32_t n, int32_t* idx,
                        void* stream);

/* The opposite ranking (Table 3, the strategy that caches the
 * minimum-similarity tokens): idx[slot, 0..n) = the n tokens of the slot
 * with the largest score (NaN ranks last, ties to the lower index),
 * ascending.  seq <= 4096. */
mar_status mar_k_select_most_similar(const double* scores, int32_t n_slots, int32_t seq, int32_t n,
                                     int32_t* idx, void* stream);

/* Tuning hook: force tile configuration `variant` (0 .. MAR_GEMM_VARIANTS-1)
 * for every later matrix product of the process, or -1 to restore the
 * choice by shape.  Every configuration uses the same MFMA instruction and
 * visits k in the same order, so results do not change by a single bit.
 * Not thread-safe with concurrent launches. */
#define MAR_GEMM_VARIANTS 16
mar_status mar_k_gemm_variant(int32_t variant);

#ifdef __cplusplus
}
#endif

#endif /* MAR_KERNELS_H */
