// MAR's per-token diffusion head with classifier-free guidance (the
// condition cache's unconditional rows feed its unconditional branch): the
// network, the DDPM sampler and their C ABI (include/mar_head.h).
//
// One call samples R tokens.  The conditional and the unconditional
// evaluation of every token run as one batch of 2R rows (rows [0, R)
// conditional, [R, 2R) unconditional), so each product of the network is
// one launch over 2R rows:
//   per call           gather z rows -> bf16; c = z W_z^T + b_z (fp32)
//   per sampling step  prologue: s = silu(c + e_i) (bf16), h = x W_in^T + b_in
//                      m = s W_ada^T + b_ada (every block's shift/scale/gate
//                          and the final shift/scale in one product: s does
//                          not depend on the block)
//                      per block: u = ln(h)(1 + scale) + shift (bf16);
//                          g = silu(u W1^T + b1) (bf16);
//                          h = h + gate (g W2^T + b2) (fp32, in place)
//                      out: per token, both rows' final ln-modulation and
//                          output product, the guidance mix and the DDPM
//                          update of the token's latent
// The products are the block GEMM kernel with the SILU and GATE epilogues.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <memory>
#include <mutex>
#include <new>
#include <system_error>

#include "../../include/mar_head.h"
#include "common.h"

using namespace marcache;

namespace {

mar_status hfail(mar_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  abi_fail_v(s, fmt, ap);
  va_end(ap);
  return s;
}

#define HEAD_HIP(call, what)                                                          \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) return hfail(MAR_E_DEVICE, "%s: %s", what, hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// The respaced DDPM coefficients of every sampling step i, in fp64 on one
// thread (a running product over the training steps): coef[i] = (1 /
// sqrt(1 - beta_i), beta_i / sqrt(1 - abar_i), sigma_i, t_i), with t_i =
// floor(i * train_steps / steps), abar_i the product of (1 - beta) up to
// t_i, beta_i = 1 - abar_i / abar_(i-1), sigma_i^2 = beta_i (1 - abar_(i-1))
// / (1 - abar_i) and sigma_0 = 0.
__global__ void head_schedule_kernel(int steps, int train_steps, double beta_start, double beta_end,
                                     f32x4_t* __restrict__ coef) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const double step = train_steps > 1 ? (beta_end - beta_start) / (train_steps - 1) : 0.0;
  double abar = 1.0, abar_kept = 1.0;
  int next = 0;
  for (int k = 0; k < train_steps && next < steps; ++k) {
    abar *= 1.0 - (beta_start + step * k);
    while (next < steps && static_cast<long>(next) * train_steps / steps == k) {
      const double beta = 1.0 - abar / abar_kept;
      const double sigma = next == 0 ? 0.0 : sqrt(beta * (1.0 - abar_kept) / (1.0 - abar));
      coef[next] = f32x4_t{static_cast<float>(1.0 / sqrt(1.0 - beta)), static_cast<float>(beta / sqrt(1.0 - abar)),
                           static_cast<float>(sigma), static_cast<float>(k)};
      abar_kept = abar;
      ++next;
    }
  }
}

// Sinusoidal features of every sampling step's timestep, bf16 [steps, F]:
// [cos(t f_k) for k < F/2, sin(t f_k) ...], f_k = 10000^(-k / (F/2)), in
// fp64 before the rounding.
__global__ void head_phi_kernel(const f32x4_t* __restrict__ coef, int steps, int F, bf16_t* __restrict__ phi) {
  const int i = blockIdx.x;
  const int half = F / 2;
  if (i >= steps) return;
  const double t = coef[i][3];
  for (int k = threadIdx.x; k < F; k += blockDim.x) {
    const int j = k < half ? k : k - half;
    const double a = t * exp(-log(10000.0) * j / half);
    phi[static_cast<long>(i) * F + k] = f2bf(static_cast<float>(k < half ? cos(a) : sin(a)));
  }
}

__global__ void head_fill_zero_kernel(float* __restrict__ p, long n4) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n4) reinterpret_cast<f32x4_t*>(p)[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

// Rows [0, R) of `out` from y_cond[row_cond[r]], rows [R, 2R) from
// y_uncond[row_uncond[r]], rounded to bf16; an index outside [0, y_rows)
// gives a zero row.  One wave per output row.
__global__ __launch_bounds__(256) void head_gather_kernel(const float* __restrict__ yc,
                                                          const float* __restrict__ yu, int y_rows,
                                                          const int32_t* __restrict__ rc,
                                                          const int32_t* __restrict__ ru, int R, int D,
                                                          bf16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= 2 * R) return;
  const bool unc = row >= R;
  const int r = unc ? row - R : row;
  const int src = unc ? ru[r] : rc[r];
  const float* y = unc ? yu : yc;
  const bool ok = src >= 0 && src < y_rows;
  for (int c = lane * 4; c < D; c += 256) {
    f32x4_t v = ok ? *reinterpret_cast<const f32x4_t*>(y + static_cast<long>(src) * D + c) : f32x4_t{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<u32x2_t*>(out + static_cast<long>(row) * D + c) = u32x2_t{pack2bf(v[0], v[1]), pack2bf(v[2], v[3])};
  }
}

__device__ __forceinline__ float silu_h(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

// in_w [w, T] (bf16) -> in_wt [T, w] (fp32), once at init, so that the
// prologue reads four consecutive columns of one input component per load.
__global__ void head_transpose_in_kernel(const bf16_t* __restrict__ in_w, int w, int T, float* __restrict__ in_wt) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(w) * T) return;
  const int col = static_cast<int>(i / T), j = static_cast<int>(i - static_cast<long>(col) * T);
  in_wt[static_cast<long>(j) * w + col] = bf2f(in_w[i]);
}

// Per sampling step, one wave per row r of the 2R: s[r] = silu(c[r] + e)
// (bf16) and h[r] = b_in + W_in x[r mod R] (fp32), with in_wt = W_in^T
// [T, w] in fp32.  TT = T when the token width is fixed at compile time
// (16, KL-16 latents): the token's latent then sits in registers and every
// weight load of a column group is issued before its multiply-adds.
template <int TT>
__global__ __launch_bounds__(256) void head_prologue_kernel(const float* __restrict__ c,
                                                            const float* __restrict__ e,
                                                            const float* __restrict__ x,
                                                            const float* __restrict__ in_wt,
                                                            const float* __restrict__ in_b, int R, int w, int T,
                                                            bf16_t* __restrict__ s, float* __restrict__ h) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= 2 * R) return;
  const float* xr = x + static_cast<long>(row >= R ? row - R : row) * T;
  const long base = static_cast<long>(row) * w;
  float xv[TT > 0 ? TT : 1];
  if constexpr (TT > 0) {
#pragma unroll
    for (int j = 0; j < TT; j += 4) {
      const f32x4_t q = *reinterpret_cast<const f32x4_t*>(xr + j);
      xv[j] = q[0];
      xv[j + 1] = q[1];
      xv[j + 2] = q[2];
      xv[j + 3] = q[3];
    }
  }
  for (int col = lane * 4; col < w; col += 256) {
    const f32x4_t cv = *reinterpret_cast<const f32x4_t*>(c + base + col);
    const f32x4_t ev = *reinterpret_cast<const f32x4_t*>(e + col);
    f32x4_t hv = *reinterpret_cast<const f32x4_t*>(in_b + col);
    if constexpr (TT > 0) {
      f32x4_t wv[TT];
#pragma unroll
      for (int j = 0; j < TT; ++j) wv[j] = *reinterpret_cast<const f32x4_t*>(in_wt + static_cast<long>(j) * w + col);
#pragma unroll
      for (int j = 0; j < TT; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) hv[q] = fmaf(xv[j], wv[j][q], hv[q]);
    } else {
      for (int j = 0; j < T; ++j) {
        const float xj = xr[j];
        const f32x4_t wv = *reinterpret_cast<const f32x4_t*>(in_wt + static_cast<long>(j) * w + col);
#pragma unroll
        for (int q = 0; q < 4; ++q) hv[q] = fmaf(xj, wv[q], hv[q]);
      }
    }
    *reinterpret_cast<u32x2_t*>(s + base + col) =
        u32x2_t{pack2bf(silu_h(cv[0] + ev[0]), silu_h(cv[1] + ev[1])), pack2bf(silu_h(cv[2] + ev[2]), silu_h(cv[3] + ev[3]))};
    *reinterpret_cast<f32x4_t*>(h + base + col) = hv;
  }
}

// Rows of the head are held 4 columns per lane per group: group k of lane
// l is columns 4 l + 256 k .. + 3.  EXACT: the width is exactly 256 G, so
// no group needs a bounds check (1024, 1280, 1536 = 256 x 4, 5, 6);
// otherwise groups past the width are skipped.
template <int G, bool EXACT>
__device__ __forceinline__ bool group_in(int lane, int k, int w) {
  return EXACT || lane * 4 + 256 * k < w;
}

__device__ __forceinline__ float bf_lo(uint32_t a) { return __uint_as_float(a << 16); }
__device__ __forceinline__ float bf_hi(uint32_t a) { return __uint_as_float(a & 0xFFFF0000u); }

// Row statistics (mean, 1 / sqrt(var + eps)) of a row held in v.
template <int G, bool EXACT>
__device__ __forceinline__ void row_stats(const f32x4_t (&v)[G], int lane, int w, float eps, float& mean,
                                          float& rstd) {
  float sum = 0.f;
#pragma unroll
  for (int k = 0; k < G; ++k)
    if (group_in<G, EXACT>(lane, k, w)) sum += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
  mean = wave_sum(sum) / static_cast<float>(w);
  float sq = 0.f;
#pragma unroll
  for (int k = 0; k < G; ++k)
    if (group_in<G, EXACT>(lane, k, w))
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float d = v[k][q] - mean;
        sq = fmaf(d, d, sq);
      }
  rstd = __builtin_amdgcn_rsqf(wave_sum(sq) / static_cast<float>(w) + eps);
}

// v <- ln(v) (1 + scale) + shift for row `row` of h, with the shift and
// scale at columns shift_off / scale_off of the modulation row mr.  Every
// load (the row, then the shift and scale) is issued before the first
// reduction.
template <int G, bool EXACT>
__device__ __forceinline__ void load_lnmod(const float* __restrict__ hrow, const bf16_t* __restrict__ mr,
                                           int shift_off, int scale_off, int lane, int w, float eps,
                                           f32x4_t (&v)[G]) {
  u32x2_t sh[G], sc[G];
#pragma unroll
  for (int k = 0; k < G; ++k) {
    const int col = lane * 4 + 256 * k;
    if (group_in<G, EXACT>(lane, k, w)) {
      v[k] = *reinterpret_cast<const f32x4_t*>(hrow + col);
      sh[k] = *reinterpret_cast<const u32x2_t*>(mr + shift_off + col);
      sc[k] = *reinterpret_cast<const u32x2_t*>(mr + scale_off + col);
    } else {
      v[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      sh[k] = sc[k] = u32x2_t{0u, 0u};
    }
  }
  float mean, rstd;
  row_stats<G, EXACT>(v, lane, w, eps, mean, rstd);
#pragma unroll
  for (int k = 0; k < G; ++k) {
    v[k][0] = fmaf((v[k][0] - mean) * rstd, 1.0f + bf_lo(sc[k][0]), bf_lo(sh[k][0]));
    v[k][1] = fmaf((v[k][1] - mean) * rstd, 1.0f + bf_hi(sc[k][0]), bf_hi(sh[k][0]));
    v[k][2] = fmaf((v[k][2] - mean) * rstd, 1.0f + bf_lo(sc[k][1]), bf_lo(sh[k][1]));
    v[k][3] = fmaf((v[k][3] - mean) * rstd, 1.0f + bf_hi(sc[k][1]), bf_hi(sh[k][1]));
  }
}

// u[r] = ln(h[r]) (1 + scale[r]) + shift[r] (bf16), one wave per row; the
// shift and scale are columns [shift_off, +w) and [scale_off, +w) of the
// modulation rows m [rows, ld] (bf16).
template <int G, bool EXACT>
__global__ __launch_bounds__(256) void head_lnmod_kernel(const float* __restrict__ h,
                                                         const bf16_t* __restrict__ m, int ld, int shift_off,
                                                         int scale_off, int rows, int w, float eps,
                                                         bf16_t* __restrict__ u) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const long base = static_cast<long>(row) * w;
  f32x4_t v[G];
  load_lnmod<G, EXACT>(h + base, m + static_cast<long>(row) * ld, shift_off, scale_off, lane, w, eps, v);
#pragma unroll
  for (int k = 0; k < G; ++k) {
    const int col = lane * 4 + 256 * k;
    if (group_in<G, EXACT>(lane, k, w))
      *reinterpret_cast<u32x2_t*>(u + base + col) = u32x2_t{pack2bf(v[k][0], v[k][1]), pack2bf(v[k][2], v[k][3])};
  }
}

// One workgroup of two waves per token r: wave p takes row r + p R (p = 0
// the conditional row, 1 the unconditional one): its final ln-modulation
// and output product.  Then the guided prediction eps = eps_u + s (eps_c -
// eps_u) and the DDPM update of x[r] with the coefficients of sampling step
// i and the draw xi_i[r] (not read when sigma_i = 0).
//
// Each lane forms partial sums of all output components over its columns;
// with T <= 16 they are summed across the wave by a reduce-scatter: four
// halving exchanges (lane distance 32, 16, 8, 4) each keep half of the
// components and add the partner's copy of that half, then two full
// exchanges (distance 2, 1) complete the sum, leaving component
// o = bits 5..2 of the lane in every lane of its group of four (a fixed
// tree: deterministic).  Wider tokens take one wave reduction per
// component.
template <int G, bool EXACT>
__global__ __launch_bounds__(128) void head_out_kernel(const float* __restrict__ h,
                                                       const bf16_t* __restrict__ m, int ld, int shift_off,
                                                       int scale_off, const bf16_t* __restrict__ out_w,
                                                       const float* __restrict__ out_b, const f32x4_t* __restrict__ coef,
                                                       int i, const float* __restrict__ xi, int R, int w, int T,
                                                       float eps_ln, float scale, float* __restrict__ x,
                                                       float* __restrict__ traj, float* __restrict__ eps_out) {
  __shared__ float eps_sh[2][64];
  const int lane = threadIdx.x & 63;
  const int p = threadIdx.x >> 6;
  const int r = blockIdx.x;
  constexpr int TB = 16;  // components reduced by the butterfly
  const long row = r + static_cast<long>(p) * R;
  f32x4_t v[G];
  load_lnmod<G, EXACT>(h + row * w, m + row * ld, shift_off, scale_off, lane, w, eps_ln, v);
  if (T <= TB) {
    float acc[TB];
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      float part = 0.f;
      if (t < T) {
        u32x2_t wv[G];
#pragma unroll
        for (int k = 0; k < G; ++k)
          wv[k] = group_in<G, EXACT>(lane, k, w)
                      ? *reinterpret_cast<const u32x2_t*>(out_w + static_cast<long>(t) * w + lane * 4 + 256 * k)
                      : u32x2_t{0u, 0u};
#pragma unroll
        for (int k = 0; k < G; ++k) {
          part = fmaf(v[k][0], bf_lo(wv[k][0]), part);
          part = fmaf(v[k][1], bf_hi(wv[k][0]), part);
          part = fmaf(v[k][2], bf_lo(wv[k][1]), part);
          part = fmaf(v[k][3], bf_hi(wv[k][1]), part);
        }
      }
      acc[t] = part;
    }
    // reduce-scatter: after the exchange at distance d, lanes with that bit
    // set hold the upper half of the remaining components
#pragma unroll
    for (int half = TB / 2, d = 32; half >= 1; half >>= 1, d >>= 1) {
      const bool up = (lane & d) != 0;
#pragma unroll
      for (int k = 0; k < half; ++k) {
        const float keep = up ? acc[k + half] : acc[k];
        const float send = up ? acc[k] : acc[k + half];
        acc[k] = keep + __shfl_xor(send, d, 64);
      }
    }
    float tot = acc[0];
    tot += __shfl_xor(tot, 2, 64);
    tot += __shfl_xor(tot, 1, 64);
    const int comp = (((lane >> 5) & 1) << 3) | (((lane >> 4) & 1) << 2) | (((lane >> 3) & 1) << 1) | ((lane >> 2) & 1);
    if ((lane & 3) == 0 && comp < T) eps_sh[p][comp] = tot + out_b[comp];
  } else {
    for (int t = 0; t < T; ++t) {
      float part = 0.f;
#pragma unroll
      for (int k = 0; k < G; ++k) {
        if (!group_in<G, EXACT>(lane, k, w)) continue;
        const u32x2_t wv = *reinterpret_cast<const u32x2_t*>(out_w + static_cast<long>(t) * w + lane * 4 + 256 * k);
        part = fmaf(v[k][0], bf_lo(wv[0]), part);
        part = fmaf(v[k][1], bf_hi(wv[0]), part);
        part = fmaf(v[k][2], bf_lo(wv[1]), part);
        part = fmaf(v[k][3], bf_hi(wv[1]), part);
      }
      const float tot = wave_sum(part) + out_b[t];
      if (lane == t) eps_sh[p][t] = tot;
    }
  }
  __syncthreads();
  if (p == 0 && lane < T) {
    const f32x4_t cf = coef[i];
    const float ec = eps_sh[0][lane], eu = eps_sh[1][lane];
    const float eg = fmaf(scale, ec - eu, eu);
    const long at = static_cast<long>(r) * T + lane;
    const float xv = x[at];
    float nx = cf[0] * fmaf(-cf[1], eg, xv);
    if (cf[2] != 0.f) nx = fmaf(cf[2], xi[static_cast<long>(i) * R * T + at], nx);
    x[at] = nx;
    if (traj) traj[at] = nx;
    if (eps_out) eps_out[at] = eg;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// Handle and C ABI
// ---------------------------------------------------------------------------

// Scratch of one call: 2R rows of the network's activations (R tokens) and
// the R latents.
struct HeadScratch {
  bf16_t* a0;  // [2R, cond_dim]
  float* c;    // [2R, w]
  bf16_t* s;   // [2R, w]
  bf16_t* m;   // [2R, n_mod w]
  float* h;    // [2R, w]
  bf16_t* u;   // [2R, w]
  bf16_t* g;   // [2R, w]
  float* x;    // [R, T]
};

struct mar_head {
  mar_head_dims d;
  int n_mod;
  // weights (matrices bf16, biases fp32)
  void *z_w, *t1_w, *t2_w, *in_w, *ada_w, *fc1_w, *fc2_w, *out_w;
  float *z_b, *t1_b, *t2_b, *in_b, *ada_b, *fc1_b, *fc2_b, *out_b;
  float* in_wt;    // [T, w] the input product's weights, transposed, fp32
  float* e;        // [steps, w] time embeddings
  f32x4_t* coef;   // [steps] DDPM coefficients
  bf16_t* phi;     // [steps, freq] (init only)
  bf16_t* t1o;     // [steps, w] (init only)
  HeadScratch sc;  // in the workspace, for up to max_rows tokens
};

namespace {

mar_status check_head_dims(const mar_head_dims* d) {
  if (!d) return hfail(MAR_E_ARG, "dims is NULL");
  if (d->dtype != MAR_BF16) return hfail(MAR_E_ARG, "the diffusion head runs in bf16 (dtype %d)", d->dtype);
  if (d->width < 64 || d->width % 64 || d->width > 4096)
    return hfail(MAR_E_SHAPE, "width %d must be a multiple of 64 in [64, 4096]", d->width);
  if (d->depth < 1) return hfail(MAR_E_SHAPE, "depth must be >= 1");
  if (d->cond_dim < 64 || d->cond_dim % 64 || d->cond_dim > 4096)
    return hfail(MAR_E_SHAPE, "cond_dim %d must be a multiple of 64 in [64, 4096]", d->cond_dim);
  if (d->token_dim < 1 || d->token_dim > 64) return hfail(MAR_E_SHAPE, "token_dim must be in [1, 64]");
  if (d->freq_dim < 64 || d->freq_dim % 64 || d->freq_dim > 1024)
    return hfail(MAR_E_SHAPE, "freq_dim must be a multiple of 64 in [64, 1024]");
  if (d->steps < 1 || d->train_steps < d->steps || d->train_steps > 100000)
    return hfail(MAR_E_SHAPE, "need 1 <= steps <= train_steps <= 100000");
  if (!(d->beta_start > 0.f) || !(d->beta_end >= d->beta_start) || !(d->beta_end < 1.f))
    return hfail(MAR_E_ARG, "need 0 < beta_start <= beta_end < 1");
  if (!(d->ln_eps > 0.f)) return hfail(MAR_E_ARG, "ln_eps must be positive");
  if (d->max_rows < 1 || d->max_rows > 65536) return hfail(MAR_E_SHAPE, "max_rows must be in [1, 65536]");
  const size_t n_mod = 3 * static_cast<size_t>(d->depth) + 2;
  if (2 * static_cast<size_t>(d->max_rows) * n_mod * d->width * 4 >= (size_t(1) << 31))
    return hfail(MAR_E_SHAPE, "2 max_rows (3 depth + 2) width * 4 reaches 2 GiB (32-bit offsets)");
  return MAR_OK;
}

// Byte offsets of the scratch of a call on `rows` tokens (256-byte
// aligned, from 0, in the order of HeadScratch's fields); returns its size.
constexpr int kScratchBuffers = 8;
size_t scratch_layout(const mar_head_dims& d, size_t rows, size_t* off) {
  const size_t w = d.width, D = d.cond_dim, T = d.token_dim;
  const size_t nm = 3 * static_cast<size_t>(d.depth) + 2, R2 = 2 * rows;
  const size_t sizes[kScratchBuffers] = {R2 * D * 2, R2 * w * 4, R2 * w * 2, R2 * nm * w * 2,
                                         R2 * w * 4, R2 * w * 2, R2 * w * 2, rows * T * 4};
  size_t o = 0;
  for (int k = 0; k < kScratchBuffers; ++k) {
    off[k] = o;
    o = align_up(o + sizes[k]);
  }
  return o;
}

HeadScratch scratch_at(unsigned char* base, const size_t* off) {
  HeadScratch sc;
  sc.a0 = reinterpret_cast<bf16_t*>(base + off[0]);
  sc.c = reinterpret_cast<float*>(base + off[1]);
  sc.s = reinterpret_cast<bf16_t*>(base + off[2]);
  sc.m = reinterpret_cast<bf16_t*>(base + off[3]);
  sc.h = reinterpret_cast<float*>(base + off[4]);
  sc.u = reinterpret_cast<bf16_t*>(base + off[5]);
  sc.g = reinterpret_cast<bf16_t*>(base + off[6]);
  sc.x = reinterpret_cast<float*>(base + off[7]);
  return sc;
}

// Byte offsets of the weights and tables in the workspace (in the order of
// mar_head's fields), followed by the scratch for max_rows tokens at
// off[kTables]; returns the total.
constexpr int kTables = 21;
size_t head_layout(const mar_head_dims& d, size_t* off) {
  const size_t w = d.width, D = d.cond_dim, T = d.token_dim, F = d.freq_dim, S = d.steps;
  const size_t nm = 3 * static_cast<size_t>(d.depth) + 2, L = d.depth;
  const size_t sizes[kTables] = {
      w * D * 2, w * F * 2, w * w * 2, w * T * 2, nm * w * w * 2, L * w * w * 2, L * w * w * 2, T * w * 2,
      w * 4, w * 4, w * 4, w * 4, nm * w * 4, L * w * 4, L * w * 4, T * 4,
      S * w * 4, S * 16, S * F * 2, S * w * 2, T * w * 4};
  size_t o = 0;
  for (int k = 0; k < kTables; ++k) {
    off[k] = o;
    o = align_up(o + sizes[k]);
  }
  off[kTables] = o;
  size_t soff[kScratchBuffers];
  return o + scratch_layout(d, static_cast<size_t>(d.max_rows), soff);
}
constexpr int kHeadBuffers = kTables + 1;

template <class Kern, class... Args>
hipError_t launch_rows(Kern k, int rows, hipStream_t st, Args... args) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k, dim3((rows + 3) / 4), dim3(256), 0, st, args...);
  return hipGetLastError();
}

// ln-modulation and output kernels by the groups of 4 a lane holds
template <int G, bool EXACT>
hipError_t lnmod_as(const mar_head* hd, const HeadScratch& sc, int off_shift, int off_scale, int rows,
                    hipStream_t st) {
  return launch_rows(head_lnmod_kernel<G, EXACT>, rows, st, static_cast<const float*>(sc.h),
                     static_cast<const bf16_t*>(sc.m), hd->n_mod * hd->d.width, off_shift, off_scale, rows,
                     hd->d.width, hd->d.ln_eps, sc.u);
}
hipError_t launch_lnmod(const mar_head* hd, const HeadScratch& sc, int off_shift, int off_scale, int rows,
                        hipStream_t st) {
  switch (hd->d.width) {
    case 1024: return lnmod_as<4, true>(hd, sc, off_shift, off_scale, rows, st);
    case 1280: return lnmod_as<5, true>(hd, sc, off_shift, off_scale, rows, st);
    case 1536: return lnmod_as<6, true>(hd, sc, off_shift, off_scale, rows, st);
    default: break;
  }
  const int G = (hd->d.width + 255) / 256;
  if (G <= 2) return lnmod_as<2, false>(hd, sc, off_shift, off_scale, rows, st);
  if (G <= 4) return lnmod_as<4, false>(hd, sc, off_shift, off_scale, rows, st);
  if (G <= 8) return lnmod_as<8, false>(hd, sc, off_shift, off_scale, rows, st);
  return lnmod_as<16, false>(hd, sc, off_shift, off_scale, rows, st);
}
template <int G, bool EXACT>
hipError_t out_as(const mar_head* hd, const HeadScratch& sc, int i, const float* xi, int R, float scale,
                  float* traj, float* eps_out, hipStream_t st) {
  const int w = hd->d.width;
  auto kern = head_out_kernel<G, EXACT>;
  hipLaunchKernelGGL(kern, dim3(R), dim3(128), 0, st, static_cast<const float*>(sc.h),
                     static_cast<const bf16_t*>(sc.m), hd->n_mod * w, 3 * hd->d.depth * w, (3 * hd->d.depth + 1) * w,
                     static_cast<const bf16_t*>(hd->out_w), static_cast<const float*>(hd->out_b),
                     static_cast<const f32x4_t*>(hd->coef), i, xi, R, w, hd->d.token_dim, hd->d.ln_eps, scale, sc.x,
                     traj, eps_out);
  return hipGetLastError();
}
hipError_t launch_out(const mar_head* hd, const HeadScratch& sc, int i, const float* xi, int R, float scale,
                      float* traj, float* eps_out, hipStream_t st) {
  switch (hd->d.width) {
    case 1024: return out_as<4, true>(hd, sc, i, xi, R, scale, traj, eps_out, st);
    case 1280: return out_as<5, true>(hd, sc, i, xi, R, scale, traj, eps_out, st);
    case 1536: return out_as<6, true>(hd, sc, i, xi, R, scale, traj, eps_out, st);
    default: break;
  }
  const int G = (hd->d.width + 255) / 256;
  if (G <= 2) return out_as<2, false>(hd, sc, i, xi, R, scale, traj, eps_out, st);
  if (G <= 4) return out_as<4, false>(hd, sc, i, xi, R, scale, traj, eps_out, st);
  if (G <= 8) return out_as<8, false>(hd, sc, i, xi, R, scale, traj, eps_out, st);
  return out_as<16, false>(hd, sc, i, xi, R, scale, traj, eps_out, st);
}

hipError_t fill_zero(float* p, long n, hipStream_t st) {
  const long n4 = n / 4;  // every zeroed buffer holds a multiple of 4 floats
  if (n4 <= 0) return hipSuccess;
  hipLaunchKernelGGL(head_fill_zero_kernel, dim3((n4 + 255) / 256), dim3(256), 0, st, p, n4);
  return hipGetLastError();
}

hipError_t gemm(const void* a, const void* w, int M, int N, int K, const EpiArgs& e, hipStream_t st) {
  return launch_gemm(DT_BF16, a, w, M, N, K, e, st);
}

mar_status head_init(const mar_head_dims* dims, const mar_head_weights* W, void* workspace, size_t bytes,
                     void* stream, mar_head** out) {
  if (!out) return hfail(MAR_E_ARG, "out is NULL");
  *out = nullptr;
  mar_status s = check_head_dims(dims);
  if (s != MAR_OK) return s;
  if (!W) return hfail(MAR_E_ARG, "weights is NULL");
  const void* ptrs[] = {W->z_w, W->z_b, W->t1_w, W->t1_b, W->t2_w, W->t2_b, W->in_w, W->in_b,
                        W->ada_w, W->ada_b, W->fc1_w, W->fc1_b, W->fc2_w, W->fc2_b, W->out_w, W->out_b};
  for (const void* p : ptrs)
    if (!p) return hfail(MAR_E_ARG, "a weight pointer is NULL");
  if (!workspace) return hfail(MAR_E_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign) return hfail(MAR_E_WORKSPACE, "workspace must be 256-byte aligned");
  size_t off[kHeadBuffers];
  const size_t need = head_layout(*dims, off);
  if (bytes < need) return hfail(MAR_E_WORKSPACE, "workspace holds %zu bytes, %zu needed", bytes, need);
  std::unique_ptr<mar_head> hd(new (std::nothrow) mar_head);
  if (!hd) return hfail(MAR_E_HOST, "out of host memory");
  const mar_head_dims& d = *dims;
  hd->d = d;
  hd->n_mod = 3 * d.depth + 2;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  void** mats[] = {&hd->z_w, &hd->t1_w, &hd->t2_w, &hd->in_w, &hd->ada_w, &hd->fc1_w, &hd->fc2_w, &hd->out_w};
  float** vecs[] = {&hd->z_b, &hd->t1_b, &hd->t2_b, &hd->in_b, &hd->ada_b, &hd->fc1_b, &hd->fc2_b, &hd->out_b};
  for (int k = 0; k < 8; ++k) *mats[k] = ws + off[k];
  for (int k = 0; k < 8; ++k) *vecs[k] = reinterpret_cast<float*>(ws + off[8 + k]);
  hd->e = reinterpret_cast<float*>(ws + off[16]);
  hd->coef = reinterpret_cast<f32x4_t*>(ws + off[17]);
  hd->phi = reinterpret_cast<bf16_t*>(ws + off[18]);
  hd->t1o = reinterpret_cast<bf16_t*>(ws + off[19]);
  hd->in_wt = reinterpret_cast<float*>(ws + off[20]);
  size_t soff[kScratchBuffers];
  scratch_layout(d, static_cast<size_t>(d.max_rows), soff);
  hd->sc = scratch_at(ws + off[kTables], soff);

  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t w = d.width, D = d.cond_dim, T = d.token_dim, F = d.freq_dim, L = d.depth, nm = hd->n_mod;
  struct Cp { void* dst; const void* src; size_t bytes; } cps[] = {
      {hd->z_w, W->z_w, w * D * 2},       {hd->t1_w, W->t1_w, w * F * 2},    {hd->t2_w, W->t2_w, w * w * 2},
      {hd->in_w, W->in_w, w * T * 2},     {hd->ada_w, W->ada_w, nm * w * w * 2},
      {hd->fc1_w, W->fc1_w, L * w * w * 2}, {hd->fc2_w, W->fc2_w, L * w * w * 2}, {hd->out_w, W->out_w, T * w * 2},
      {hd->z_b, W->z_b, w * 4},           {hd->t1_b, W->t1_b, w * 4},        {hd->t2_b, W->t2_b, w * 4},
      {hd->in_b, W->in_b, w * 4},         {hd->ada_b, W->ada_b, nm * w * 4}, {hd->fc1_b, W->fc1_b, L * w * 4},
      {hd->fc2_b, W->fc2_b, L * w * 4},   {hd->out_b, W->out_b, T * 4}};
  for (const Cp& cp : cps) HEAD_HIP(hipMemcpyAsync(cp.dst, cp.src, cp.bytes, hipMemcpyDeviceToDevice, st), "weight copy");
  // the sampler's coefficients and the time embedding of every step
  hipLaunchKernelGGL(head_schedule_kernel, dim3(1), dim3(64), 0, st, d.steps, d.train_steps,
                     static_cast<double>(d.beta_start), static_cast<double>(d.beta_end), hd->coef);
  HEAD_HIP(hipGetLastError(), "schedule");
  hipLaunchKernelGGL(head_phi_kernel, dim3(d.steps), dim3(256), 0, st, static_cast<const f32x4_t*>(hd->coef), d.steps,
                     d.freq_dim, hd->phi);
  HEAD_HIP(hipGetLastError(), "time features");
  EpiArgs e1{};
  e1.kind = EPI_SILU;
  e1.bias = hd->t1_b;
  e1.out = hd->t1o;
  HEAD_HIP(gemm(hd->phi, hd->t1_w, d.steps, d.width, d.freq_dim, e1, st), "time embedding (first product)");
  HEAD_HIP(fill_zero(hd->e, static_cast<long>(d.steps) * d.width, st), "zero fill");
  EpiArgs e2{};
  e2.kind = EPI_RESIDUAL;
  e2.bias = hd->t2_b;
  e2.out = hd->e;
  e2.resid = hd->e;
  HEAD_HIP(gemm(hd->t1o, hd->t2_w, d.steps, d.width, d.width, e2, st), "time embedding (second product)");
  {
    const long n = static_cast<long>(d.width) * d.token_dim;
    hipLaunchKernelGGL(head_transpose_in_kernel, dim3((n + 255) / 256), dim3(256), 0, st,
                       static_cast<const bf16_t*>(hd->in_w), d.width, d.token_dim, hd->in_wt);
    HEAD_HIP(hipGetLastError(), "input weights");
  }
  *out = hd.release();
  return MAR_OK;
}

// Arguments of a call, checked on the host (rows against the caller's
// limit, which the scratch behind the call must hold).
mar_status check_sample(const mar_head* hd, const float* yc, const float* yu, int32_t y_rows, const int32_t* rc,
                        const int32_t* ru, int32_t R, int32_t max_R, const float* x_init, const float* xi,
                        float scale, float* x_out, float* traj, float* eps_out) {
  if (!hd) return hfail(MAR_E_ARG, "head is NULL");
  if (R < 0 || R > max_R) return hfail(MAR_E_ARG, "rows %d outside [0, %d]", R, max_R);
  if (R == 0) return MAR_OK;
  if (!yc || !yu || !rc || !ru || !x_init || !xi || !x_out) return hfail(MAR_E_ARG, "NULL pointer");
  if (y_rows < 1) return hfail(MAR_E_ARG, "y_rows must be >= 1");
  const void* al[] = {yc, yu, x_init, xi, x_out, traj ? traj : x_out, eps_out ? eps_out : x_out};
  for (const void* p : al)
    if (!aligned16(p)) return hfail(MAR_E_ARG, "float buffers must be 16-byte aligned");
  if (!std::isfinite(scale)) return hfail(MAR_E_ARG, "scale must be finite");
  {
    hipError_t e = hipPeekAtLastError();
    if (e != hipSuccess) return hfail(MAR_E_DEVICE, "earlier device error: %s", hipGetErrorString(e));
  }
  return MAR_OK;
}

// The sampler over R >= 1 tokens with the scratch `sc` (checked arguments).
mar_status head_sample(const mar_head* hd, const HeadScratch& sc, const float* yc, const float* yu, int32_t y_rows,
                       const int32_t* rc, const int32_t* ru, int32_t R, const float* x_init, const float* xi,
                       float scale, float* x_out, float* traj, float* eps_out, void* stream) {
  const mar_head_dims& d = hd->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int w = d.width, D = d.cond_dim, T = d.token_dim, R2 = 2 * R, nm = hd->n_mod;
  const size_t xbytes = static_cast<size_t>(R) * T * sizeof(float);
  HEAD_HIP(launch_rows(head_gather_kernel, R2, st, yc, yu, static_cast<int>(y_rows), rc, ru, static_cast<int>(R), D,
                       sc.a0),
           "gather");
  HEAD_HIP(fill_zero(sc.c, static_cast<long>(R2) * w, st), "zero fill");
  EpiArgs ec{};
  ec.kind = EPI_RESIDUAL;
  ec.bias = hd->z_b;
  ec.out = sc.c;
  ec.resid = sc.c;
  HEAD_HIP(gemm(sc.a0, hd->z_w, R2, w, D, ec, st), "conditioning product");
  HEAD_HIP(hipMemcpyAsync(sc.x, x_init, xbytes, hipMemcpyDeviceToDevice, st), "latent copy");
  if (traj) HEAD_HIP(hipMemcpyAsync(traj, x_init, xbytes, hipMemcpyDeviceToDevice, st), "trajectory copy");
  for (int j = 0; j < d.steps; ++j) {
    const int i = d.steps - 1 - j;
    HEAD_HIP(launch_rows(T == 16 ? head_prologue_kernel<16> : head_prologue_kernel<0>, R2, st,
                         static_cast<const float*>(sc.c),
                         static_cast<const float*>(hd->e + static_cast<long>(i) * w), static_cast<const float*>(sc.x),
                         static_cast<const float*>(hd->in_wt), static_cast<const float*>(hd->in_b), static_cast<int>(R),
                         w, T, sc.s, sc.h),
             "prologue");
    EpiArgs em{};
    em.kind = EPI_BIAS;
    em.bias = hd->ada_b;
    em.out = sc.m;
    HEAD_HIP(gemm(sc.s, hd->ada_w, R2, nm * w, w, em, st), "modulation product");
    for (int k = 0; k < d.depth; ++k) {
      HEAD_HIP(launch_lnmod(hd, sc, 3 * k * w, (3 * k + 1) * w, R2, st), "ln-modulation");
      EpiArgs e1{};
      e1.kind = EPI_SILU;
      e1.bias = hd->fc1_b + static_cast<long>(k) * w;
      e1.out = sc.g;
      HEAD_HIP(gemm(sc.u, static_cast<const bf16_t*>(hd->fc1_w) + static_cast<long>(k) * w * w, R2, w, w, e1, st),
               "block first product");
      EpiArgs e2{};
      e2.kind = EPI_GATE;
      e2.bias = hd->fc2_b + static_cast<long>(k) * w;
      e2.out = sc.h;
      e2.resid = sc.h;
      e2.gate = sc.m + static_cast<long>(3 * k + 2) * w;
      e2.gate_ld = nm * w;
      HEAD_HIP(gemm(sc.g, static_cast<const bf16_t*>(hd->fc2_w) + static_cast<long>(k) * w * w, R2, w, w, e2, st),
               "block second product");
    }
    float* tj = traj ? traj + static_cast<long>(j + 1) * R * T : nullptr;
    float* ej = eps_out ? eps_out + static_cast<long>(j) * R * T : nullptr;
    HEAD_HIP(launch_out(hd, sc, i, xi, R, scale, tj, ej, st), "output and sampler step");
  }
  HEAD_HIP(hipMemcpyAsync(x_out, sc.x, xbytes, hipMemcpyDeviceToDevice, st), "latent copy");
  return MAR_OK;
}

// ---------------------------------------------------------------------------
// Scratch of mar_head_sample_noalloc: one file-scope array per GPU, for
// callers that cannot allocate device memory.  In host code `scratch` names
// a host-side stand-in; the array's device address comes from
// hipGetSymbolAddress, resolved once per device (at init, else at the
// first call on that device) and kept in kScratchPtr.
// ---------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.
mar_status static_scratch(void** out) {
  int dev = -1;
  HEAD_HIP(hipGetDevice(&dev), "current device");
  if (dev < 0 || dev >= kMaxDevices) return hfail(MAR_E_DEVICE, "device %d beyond the scratch table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HEAD_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "scratch address");
    if (!p) return hfail(MAR_E_DEVICE, "scratch address is NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MAR_OK;
}

}  // namespace

extern "C" {

size_t mar_head_workspace_bytes(const mar_head_dims* dims) {
  abi_clear_error();
  if (check_head_dims(dims) != MAR_OK) return 0;
  size_t off[kHeadBuffers];
  return head_layout(*dims, off);
}

mar_status mar_head_init(const mar_head_dims* dims, const mar_head_weights* weights, void* workspace,
                         size_t workspace_bytes, void* stream, mar_head** out) {
  abi_clear_error();
  try {
    mar_status s = head_init(dims, weights, workspace, workspace_bytes, stream, out);
    if (s != MAR_OK) return s;
    void* p = nullptr;
    s = static_scratch(&p);  // the allocation-free entry point's array, resolved here once per device
    if (s != MAR_OK) {
      delete *out;
      *out = nullptr;
    }
    return s;
  } catch (const std::bad_alloc&) {
    return hfail(MAR_E_HOST, "out of host memory");
  } catch (const std::system_error&) {
    return hfail(MAR_E_HOST, "lock failed");
  }
}

mar_status mar_head_sample(mar_head* head, const float* y_cond, const float* y_uncond, int32_t y_rows,
                           const int32_t* row_cond, const int32_t* row_uncond, int32_t rows, const float* x_init,
                           const float* xi, float scale, float* x_out, float* trajectory, float* eps_out,
                           void* stream) {
  abi_clear_error();
  mar_status s = check_sample(head, y_cond, y_uncond, y_rows, row_cond, row_uncond, rows,
                              head ? head->d.max_rows : 0, x_init, xi, scale, x_out, trajectory, eps_out);
  if (s != MAR_OK || rows == 0) return s;
  return head_sample(head, head->sc, y_cond, y_uncond, y_rows, row_cond, row_uncond, rows, x_init, xi, scale, x_out,
                     trajectory, eps_out, stream);
}

mar_status mar_head_sample_noalloc(mar_head* head, const float* y_cond, const float* y_uncond, int32_t y_rows,
                                   const int32_t* row_cond, const int32_t* row_uncond, int32_t rows,
                                   const float* x_init, const float* xi, float scale, float* x_out,
                                   float* trajectory, float* eps_out, void* stream) {
  abi_clear_error();
  mar_status s = check_sample(head, y_cond, y_uncond, y_rows, row_cond, row_uncond, rows, 65536, x_init, xi, scale,
                              x_out, trajectory, eps_out);
  if (s != MAR_OK || rows == 0) return s;
  size_t off[kScratchBuffers];
  const size_t need = scratch_layout(head->d, static_cast<size_t>(rows), off);
  if (need > kStaticScratchBytes)
    return hfail(MAR_E_SHAPE, "%d rows need %zu bytes of scratch; the static array holds %zu", rows, need,
                 kStaticScratchBytes);
  void* base = nullptr;
  try {
    s = static_scratch(&base);
  } catch (const std::system_error&) {
    return hfail(MAR_E_HOST, "lock failed");
  }
  if (s != MAR_OK) return s;
  return head_sample(head, scratch_at(static_cast<unsigned char*>(base), off), y_cond, y_uncond, y_rows, row_cond,
                     row_uncond, rows, x_init, xi, scale, x_out, trajectory, eps_out, stream);
}

mar_status mar_head_destroy(mar_head* head) {
  delete head;
  return MAR_OK;
}

}  // extern "C"
