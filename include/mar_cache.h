/*
 * mar_cache.h - C ABI of the cached MAR transformer step on one MI355X GPU.
 *
 * LazyMAR (Yan et al., "Accelerating Masked Autoregressive Models via
 * Feature Caching", ICCV 2025) speeds up a masked-autoregressive image
 * generator by reusing work between adjacent decoding steps:
 *
 *  - token cache (Sec. 3.2, Eq. 8-9): the first P blocks run on every token;
 *    the cosine similarity between this step's and the previous step's value
 *    rows of block P-1 picks the N least similar tokens; blocks P..L-1
 *    compute only those rows, every other row is taken from the cache, and
 *    the fresh rows are written back into it;
 *  - condition cache (Sec. 3.2, Eq. 10): on a refresh step both guidance
 *    pathways run and their residual is stored; on later steps only the
 *    conditional pathway runs and the unconditional output is recovered
 *    from the stored residual;
 *  - periodic refresh (Sec. 1, Fig. 3): every tau steps a full step
 *    recomputes everything and refills both caches.
 *
 * The library runs all of this in hand-written HIP kernels for gfx950.  The
 * caller owns every device buffer, including one workspace that holds the
 * repacked weights, the per-block key/value caches, the scoring reference,
 * the output cache, the guidance residual and the scratch of a step; the
 * library never allocates device memory.
 *
 * Conventions for every call:
 *  - Pointers named "device" must point to GPU memory of the current HIP
 *    device; all are row-major and densely packed.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Work is
 *    enqueued asynchronously; outputs are valid once the stream reaches the
 *    enqueued work.  One handle must not be used on two streams at once,
 *    nor from two host threads at once.
 *  - Every argument and every state precondition is checked on the host
 *    before anything is enqueued: a call that returns an error has no
 *    effect on any buffer or on the handle's state.  mar_last_error() then
 *    holds a message for the calling thread.
 *  - A fault of an already enqueued kernel is reported by the HIP runtime
 *    and surfaces as MAR_E_DEVICE from a later call.
 *  - No C++ exception crosses this interface.
 */
#ifndef MAR_CACHE_H
#define MAR_CACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mar_cache mar_cache; /* opaque handle */

typedef enum {
  MAR_OK = 0,
  MAR_E_ARG = -1,       /* null pointer, value out of range */
  MAR_E_SHAPE = -2,     /* dimensions the kernels do not support */
  MAR_E_STATE = -3,     /* cached step before a full step, reuse before store */
  MAR_E_WORKSPACE = -4, /* workspace too small or misaligned */
  MAR_E_DEVICE = -5,    /* HIP runtime error (launch failure, earlier fault) */
  MAR_E_HOST = -6       /* host memory exhausted (handle or profiler bookkeeping) */
} mar_status;

/* Storage type of activations, weights and the key/value caches.  Matrix
 * products always accumulate in fp32; the residual stream, LayerNorm
 * statistics, the output cache and the guidance residual are fp32. */
typedef enum { MAR_F32 = 0, MAR_BF16 = 1 } mar_dtype;

typedef enum {
  /* Refresh / warm-up step (Sec. 1 "periodic cache-reuse-refreshment",
   * Fig. 3): every block on every row; fills the key/value caches of blocks
   * P..L-1, the scoring reference and the output cache of the slots, and
   * marks them filled. */
  MAR_FULL = 0,
  /* Token-cached step (Sec. 3.2, Eq. 8-9): blocks 0..P-1 on every row, the
   * similarity-based selection of n_recompute rows per slot, blocks
   * P..L-1 on those rows only. */
  MAR_TOKEN_CACHED = 1,
  /* As MAR_TOKEN_CACHED, but the computed rows are given by the caller
   * (host array, see mar_step) instead of the similarity ranking, as in the
   * random / token-type strategies the paper compares against (Table 3). */
  MAR_TOKEN_GIVEN = 2,
  /* As MAR_TOKEN_CACHED with the opposite ranking: the n_recompute MOST
   * similar rows are computed and the least similar ones taken from the
   * cache (Table 3, the strategy that caches the minimum-similarity
   * tokens). */
  MAR_TOKEN_CACHED_MOST_SIMILAR = 3
} mar_mode;

typedef enum {
  MAR_CFG_STORE = 0, /* both pathways computed: store C = u - c (Eq. 10) */
  MAR_CFG_REUSE = 1  /* conditional pathway only: u_hat = c + C (Eq. 10) */
} mar_cfg_op;

/* What the similarity of Eq. (8) compares, step to step (Sec. 4.4). */
typedef enum {
  MAR_SCORE_VALUES = 0,  /* the self-attention value rows of block P-1 (of
                            block 0, formed from x, when P = 0): the paper's
                            choice */
  MAR_SCORE_FEATURES = 1 /* the features: block P-1's output rows (fp32), or
                            the step input x when P = 0 */
} mar_score_source;

/* Shape of a stack of identical pre-LN bidirectional blocks:
 *   h = h + W_o MHA(LN1 h) + b_o ;  h = h + W_2 GELU(W_1 LN2 h + b_1) + b_2
 * with exact-erf GELU, biased-variance LayerNorm, no attention mask.
 * Supported: d_model % n_heads == 0, d_head = d_model / n_heads a multiple
 * of 16 and at most 128, d_model and d_mlp multiples of 64, 1 <= seq_len <=
 * 4096, d_model <= 2048, max_slots >= 1, 0 <= full_prefix < n_layers, and
 * max_slots * seq_len * max(3 d_model, d_mlp) * 4 < 2^31 (the kernels
 * address each operand and output with 32-bit byte offsets; MAR-H shapes,
 * seq_len 320 and d_mlp 5120, allow up to 327 slots).
 * Zero-initialize, then set the fields: the trailing options default to the
 * paper's method. */
typedef struct {
  int32_t n_layers;     /* L */
  int32_t d_model;      /* D */
  int32_t n_heads;      /* H */
  int32_t d_mlp;        /* F */
  int32_t seq_len;      /* S: buffer/class rows + image-token rows */
  int32_t max_slots;    /* sequence slots held by the caches */
  int32_t full_prefix;  /* P: blocks always computed on every row (paper: 3) */
  int32_t dtype;        /* mar_dtype */
  float ln_eps;         /* LayerNorm epsilon */
  int32_t score_source; /* mar_score_source */
  int32_t fresh_kv;     /* 0: at block P the keys/values of the rows that
                           are not computed come from the cache (Eq. 9);
                           1: they are recomputed for every row from this
                           step's block P-1 output (one key/value product
                           over all rows per cached step) */
} mar_dims;

/* Device pointers to the parameters of one block, nn.Linear layout
 * ([out, in], row-major).  Matrices are in `dtype`; LayerNorm gains/shifts
 * and biases are fp32.  qkv_w is [3D, D] with the query, key and value
 * projections stacked in that order; qkv_b is [3D]; proj_w [D, D];
 * fc1_w [F, D]; fc2_w [D, F]. */
typedef struct {
  const void *ln1_w, *ln1_b, *qkv_w, *qkv_b, *proj_w, *proj_b;
  const void *ln2_w, *ln2_b, *fc1_w, *fc1_b, *fc2_w, *fc2_b;
} mar_block_weights;

/* Bytes of workspace mar_cache_init needs for `dims` (0 if the dimensions
 * are not supported; mar_last_error() then says why). */
size_t mar_workspace_bytes(const mar_dims* dims);

/* Create a handle over a caller-allocated device workspace (256-byte
 * aligned, at least mar_workspace_bytes(dims) bytes) and copy the weights of
 * the n_layers blocks (host array `blocks` of device pointers) into it on
 * `stream`.  The caller may release its weight buffers once the stream has
 * passed this call.  The workspace must stay allocated, and must not be
 * written by the caller, until mar_cache_destroy.  All slots start unfilled
 * and no guidance residual is stored. */
mar_status mar_cache_init(const mar_dims* dims, const mar_block_weights* blocks,
                          void* workspace, size_t workspace_bytes, void* stream,
                          mar_cache** out);

/* One transformer step for the consecutive slots [slot0, slot0 + n_slots).
 *
 *  x            device [n_slots, S, D] in `dtype`, 16-byte aligned: this
 *               step's block-0 input.
 *  y            device [n_slots, S, D] fp32 or NULL: receives the output of
 *               block L-1 for every row (computed rows fresh, the others
 *               from the output cache; Eq. 9).  The same values stay in the
 *               output cache, see mar_output.
 *  mode         mar_mode.  The cached modes (MAR_TOKEN_CACHED,
 *               MAR_TOKEN_GIVEN, MAR_TOKEN_CACHED_MOST_SIMILAR) need every
 *               slot of the range filled by an earlier MAR_FULL (else
 *               MAR_E_STATE).
 *  n_recompute  N, rows computed per slot in blocks P..L-1 (0 <= N <= S);
 *               ignored by MAR_FULL.
 *  sel_idx      MAR_TOKEN_CACHED / MAR_TOKEN_CACHED_MOST_SIMILAR: device
 *               [n_slots, N] int32 or NULL; receives the computed rows of
 *               each slot in ascending token order.
 *               MAR_TOKEN_GIVEN: HOST [n_slots, N] int32, required; each
 *               slot's rows strictly ascending in [0, S) (else MAR_E_ARG);
 *               it must stay unchanged until the stream has passed this
 *               call.  Ignored by MAR_FULL.
 *
 * Selection (MAR_TOKEN_CACHED): per slot, the N rows whose value rows of
 * block P-1 (of block 0, formed from x, when P = 0; the features instead
 * with MAR_SCORE_FEATURES) have the smallest fp64 cosine similarity to the
 * slot's previous step; ties to the lower index, NaN last.
 * MAR_TOKEN_CACHED_MOST_SIMILAR: the N largest similarities, ties to the
 * lower index, NaN last.
 * Every mode replaces the slot's scoring reference with this step's value
 * rows (features). */
mar_status mar_step(mar_cache* cache, const void* x, float* y, int32_t slot0,
                    int32_t n_slots, int32_t mode, int32_t n_recompute,
                    int32_t* sel_idx, void* stream);

/* Classifier-free guidance with the condition cache (Sec. 3.1 Eq. 7,
 * Sec. 3.2 Eq. 10) for the guidance pairs [pair0, pair0 + n_pairs), each
 * [S, D] fp32 on the device:
 *   STORE:  C[p] = u - c;        guided = u + scale (c - u)   (y_uncond = u)
 *   REUSE:  u_hat = c + C[p];    guided = u_hat + scale (c - u_hat)
 * y_cond is required; y_uncond is required by STORE and ignored by REUSE;
 * guided is required; uncond_out (nullable) receives u (STORE) or u_hat
 * (REUSE).  The mix is evaluated as fmaf(scale, c - u, u) in fp32.  REUSE
 * of a pair never stored returns MAR_E_STATE.  Pairs index the residual
 * store, not slots; the store holds ceil(max_slots / 2) pairs:
 * 0 <= pair0, pair0 + n_pairs <= (max_slots + 1) / 2. */
mar_status mar_cfg_combine(mar_cache* cache, const float* y_cond,
                           const float* y_uncond, int32_t pair0, int32_t n_pairs,
                           int32_t op, float scale, float* guided,
                           float* uncond_out, void* stream);

/* Device pointer to the output cache [max_slots, S, D] fp32 inside the
 * workspace (valid until mar_cache_destroy; rows change with every step). */
const float* mar_output(const mar_cache* cache);

/* Release the handle (host memory only; the workspace stays the caller's).
 * Accepts NULL. */
mar_status mar_cache_destroy(mar_cache* cache);

/* Kernel classes of the step, for the profiler. */
typedef enum {
  MAR_PROF_QKV = 0,        /* query/key/value product (+ cache scatter) */
  MAR_PROF_PROJ = 1,       /* output projection + residual */
  MAR_PROF_FC1 = 2,        /* first MLP product + GELU */
  MAR_PROF_FC2 = 3,        /* second MLP product + residual (+ output scatter) */
  MAR_PROF_ATTENTION = 4,  /* dense and partial attention */
  MAR_PROF_LAYERNORM = 5,  /* LayerNorm, with or without the row gather */
  MAR_PROF_SCORES = 6,     /* similarity scores + reference update */
  MAR_PROF_SELECT = 7,     /* least-similar selection */
  MAR_PROF_CFG = 8,        /* guidance / condition cache */
  MAR_PROF_KINDS = 9
} mar_prof_kind;

/* Start timing every launch of kernel class `kind` made by later calls on
 * this handle: a HIP event pair is recorded around each such launch on the
 * call's stream (other classes run untouched).  A session times at most
 * 262144 launches; later launches of the class run untimed and are not
 * counted.  Restarts an open session. */
mar_status mar_profile_start(mar_cache* cache, int32_t kind);

/* End the session: waits for the recorded events and returns the summed
 * event time (ms), the number of launches, and the summed algorithmic
 * FLOPs (2 per multiply-add of the products and attention contractions)
 * and bytes (operands read once, results written once) of those launches.
 * Any output pointer may be NULL.  MAR_E_STATE without an open session. */
mar_status mar_profile_stop(mar_cache* cache, double* ms_total, int64_t* launches, double* flops,
                            double* bytes);

/* Message of the last failed call on this thread ("" if none). */
const char* mar_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MAR_CACHE_H */
