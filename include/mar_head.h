/*
 * mar_head.h - C ABI of MAR's per-token diffusion head on one MI355X GPU,
 * with classifier-free guidance fed by the condition cache.
 *
 * MAR (the model LazyMAR accelerates) samples the latent of every token
 * decoded at a decoding step with a small denoising network conditioned on
 * that token's transformer output row (Sec. 2), over 100 DDPM steps
 * (Sec. 4.1); classifier-free guidance (Eq. 7) mixes the network's
 * conditional and unconditional predictions.  LazyMAR leaves the head as it
 * is, but on its reuse steps the unconditional rows that feed it are the
 * condition cache's approximation (Eq. 10: conditional rows + the stored
 * residual; mar_cfg_combine's uncond_out).  Its cost does not depend on the
 * number of decoding steps: Table 1's constant FLOPs term.
 *
 * The paper does not give the network or the sampler; this library takes:
 *   c   = z W_z^T + b_z                       (per row, once per call)
 *   e_i = W_t2 silu(W_t1 phi(t_i) + b_t1) + b_t2   (phi: sinusoidal features
 *         [cos(t f_k), sin(t f_k)], f_k = 10000^(-k/half), of the training
 *         timestep t_i of sampling step i; computed at init)
 *   s   = silu(c + e_i);   m = s W_ada^T + b_ada   (shift/scale/gate per block,
 *                                                   final shift/scale)
 *   h   = x W_in^T + b_in
 *   block k:  h += gate_k * (silu((ln(h) (1 + scale_k) + shift_k) W1_k^T + b1_k) W2_k^T + b2_k)
 *   eps = (ln(h) (1 + scale_f) + shift_f) W_out^T + b_out
 * (ln: LayerNorm without gain and shift), and DDPM ancestral sampling on the
 * linear schedule beta in [beta_start, beta_end] over train_steps, respaced
 * to `steps` timesteps t_i = floor(i * train_steps / steps):
 *   x <- (x - beta_i / sqrt(1 - abar_i) eps) / sqrt(1 - beta_i) + sigma_i xi_i,
 *   sigma_i^2 = beta_i (1 - abar_(i-1)) / (1 - abar_i),  sigma_0 = 0,
 * for i = steps-1 down to 0, with eps = eps_u + scale (eps_c - eps_u) per
 * token (the two evaluations of a token share x).
 *
 * Storage and precision: matrices and the activations fed to products in
 * bf16, fp32 accumulation; the residual stream h, the conditioning c, the
 * latents x and the noise prediction in fp32.
 *
 * Conventions as in mar_cache.h: device pointers, row-major dense layouts,
 * asynchronous on `stream`, every argument checked on the host before any
 * enqueue (an error has no effect), MAR_E_* statuses and mar_last_error().
 */
#ifndef MAR_HEAD_H
#define MAR_HEAD_H

#include <stddef.h>
#include <stdint.h>

#include "mar_cache.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mar_head mar_head; /* opaque handle */

/* Supported: dtype MAR_BF16; width a multiple of 64, <= 4096; depth >= 1;
 * cond_dim a multiple of 64, <= 4096; token_dim in [1, 64]; freq_dim a
 * multiple of 64, <= 1024; 1 <= steps <= train_steps <= 100000;
 * 0 < beta_start <= beta_end < 1; 1 <= max_rows <= 65536 with
 * 2 max_rows (3 depth + 2) width * 4 < 2^31 (32-bit offsets of the
 * modulation product). */
typedef struct {
  int32_t width;       /* w */
  int32_t depth;       /* residual blocks */
  int32_t cond_dim;    /* width of the transformer rows z (d_model) */
  int32_t token_dim;   /* latent width of a token (16 for KL-16) */
  int32_t steps;       /* sampling steps (100) */
  int32_t train_steps; /* training timesteps of the noise schedule (1000) */
  int32_t freq_dim;    /* sinusoidal features of the time embedding (256) */
  int32_t max_rows;    /* tokens per call at most (each evaluated twice) */
  int32_t dtype;       /* mar_dtype; MAR_BF16 */
  float beta_start, beta_end;
  float ln_eps;
} mar_head_dims;

/* Device pointers, nn.Linear layout ([out, in], row-major).  Matrices in
 * `dtype`, biases fp32.  fc1_w/fc2_w hold the `depth` blocks' [w, w]
 * matrices back to back, fc1_b/fc2_b their [w] biases; ada_w is
 * [(3 depth + 2) w, w] with block k's shift, scale, gate at rows
 * (3k, 3k+1, 3k+2) w and the final shift, scale last; in_w [w, token_dim]
 * and out_w [token_dim, w] may be in `dtype` like the others. */
typedef struct {
  const void *z_w, *z_b, *t1_w, *t1_b, *t2_w, *t2_b, *in_w, *in_b, *ada_w, *ada_b;
  const void *fc1_w, *fc1_b, *fc2_w, *fc2_b, *out_w, *out_b;
} mar_head_weights;

/* Bytes of workspace mar_head_init needs (0 if `dims` is not supported;
 * mar_last_error() then says why). */
size_t mar_head_workspace_bytes(const mar_head_dims* dims);

/* Create a handle over a caller-allocated device workspace (256-byte
 * aligned, at least mar_head_workspace_bytes(dims) bytes): copies the
 * weights in and computes the time embedding of every sampling step on
 * `stream`.  The caller may release its weight buffers once the stream has
 * passed this call; the workspace stays the library's until destroy. */
mar_status mar_head_init(const mar_head_dims* dims, const mar_head_weights* weights, void* workspace,
                         size_t workspace_bytes, void* stream, mar_head** out);

/* Sample the latents of `rows` tokens (rows <= max_rows; 0 is a no-op).
 *
 *  y_cond, y_uncond  device fp32 [y_rows, cond_dim]: transformer output
 *                    rows (e.g. the output cache of mar_step, or the
 *                    unconditional rows mar_cfg_combine recovered);
 *  row_cond, row_uncond  device int32 [rows]: the row of y_cond / y_uncond
 *                    that conditions token r (the decoded tokens' rows); an
 *                    index outside [0, y_rows) reads a row of zeros;
 *  x_init            device fp32 [rows, token_dim]: the initial noise;
 *  xi                device fp32 [steps, rows, token_dim]: the Gaussian
 *                    draw of every sampling step (entry i used by step i;
 *                    entry 0 is not read);
 *  scale             guidance scale s;
 *  x_out             device fp32 [rows, token_dim]: the sampled latents;
 *  trajectory        device fp32 [steps + 1, rows, token_dim] or NULL:
 *                    entry j = x before sampling step steps-1-j (entry 0 =
 *                    x_init, entry steps = x_out);
 *  eps_out           device fp32 [steps, rows, token_dim] or NULL: entry j
 *                    = the guided noise prediction of sampling step
 *                    steps-1-j.
 * All float buffers 16-byte aligned; x_out, trajectory and eps_out must not
 * overlap the inputs. */
mar_status mar_head_sample(mar_head* head, const float* y_cond, const float* y_uncond, int32_t y_rows,
                           const int32_t* row_cond, const int32_t* row_uncond, int32_t rows,
                           const float* x_init, const float* xi, float scale, float* x_out,
                           float* trajectory, float* eps_out, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): as
 * mar_head_sample, with the same kernels and bit-identical results, but the
 * call's scratch (the activations of its 2 rows per token and the latents)
 * lives in a static array of 64 MiB per GPU instead of the handle's
 * workspace, and neither this call nor anything it calls allocates.  The
 * array's device address is resolved once per device by mar_head_init (or
 * by the first call on a device).
 * Limit: the scratch of `rows` tokens, 2 (2 cond_dim + width (14 +
 * 2 (3 depth + 2))) + 4 token_dim bytes per token plus under 2 KiB of
 * alignment, must fit 64 MiB (MAR_E_SHAPE otherwise): 387 tokens for the
 * MAR-L head (width 1280, 8 blocks, cond_dim 1024); `rows` is not bounded
 * by the handle's max_rows.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (two streams, two threads) race and give undefined results.  Each call
 * clears or overwrites all of the scratch it reads. */
mar_status mar_head_sample_noalloc(mar_head* head, const float* y_cond, const float* y_uncond, int32_t y_rows,
                                   const int32_t* row_cond, const int32_t* row_uncond, int32_t rows,
                                   const float* x_init, const float* xi, float scale, float* x_out,
                                   float* trajectory, float* eps_out, void* stream);

/* Release the handle (host memory only).  Accepts NULL. */
mar_status mar_head_destroy(mar_head* head);

#ifdef __cplusplus
}
#endif

#endif /* MAR_HEAD_H */
