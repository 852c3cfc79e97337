// Row LayerNorm of the pre-LN block, optionally gathering the rows first.
//
// One wave per row.  Each lane holds groups of 8 consecutive elements in
// registers (16-byte bf16 or 2x16-byte fp32 loads), so the statistics are a
// two-pass mean / biased variance over values already in registers, summed
// across the wave in a fixed order (DPP within rows of 16 lanes, then the
// four row sums; the result of a row never depends on which other rows are
// in the launch).  As the gather for the cached blocks
// (Eq. 9: only the computed rows enter blocks P..L-1), row m reads token
// idx[m] of its slot and the fp32 copy of that row seeds the compact
// residual stream.
#include "common.h"

namespace marcache {

template <typename TIn>
__device__ __forceinline__ void load8(const TIn* p, float* v);
template <>
__device__ __forceinline__ void load8<float>(const float* p, float* v) {
  const u32x4_t a = *reinterpret_cast<const u32x4_t*>(p);
  const u32x4_t b = *reinterpret_cast<const u32x4_t*>(p + 4);
  unpack16(a, v, static_cast<const float*>(nullptr));
  unpack16(b, v + 4, static_cast<const float*>(nullptr));
}
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* v) {
  const u32x4_t a = *reinterpret_cast<const u32x4_t*>(p);
  unpack16(a, v, static_cast<const bf16_t*>(nullptr));
}

template <typename TOut>
__device__ __forceinline__ void store8(TOut* p, const float* v);
template <>
__device__ __forceinline__ void store8<float>(float* p, const float* v) {
  u32x4_t a, b;
  for (int i = 0; i < 4; ++i) {
    a[i] = __float_as_uint(v[i]);
    b[i] = __float_as_uint(v[4 + i]);
  }
  *reinterpret_cast<u32x4_t*>(p) = a;
  *reinterpret_cast<u32x4_t*>(p + 4) = b;
}
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* p, const float* v) {
  u32x4_t a;
  for (int i = 0; i < 4; ++i) a[i] = pack2bf(v[2 * i], v[2 * i + 1]);
  *reinterpret_cast<u32x4_t*>(p) = a;
}

// G = groups of 8 elements per lane (D <= 512 G), a template parameter so
// that the row, the weight and the bias occupy exactly the registers they
// need.  The weight and bias are loaded with the row, before the first
// reduction, so their latency hides under the row's.
template <typename TIn, typename TOut, int G>
__global__ __launch_bounds__(256) void layernorm_kernel(const TIn* __restrict__ src,
                                                        const int32_t* __restrict__ idx,
                                                        int per_slot, int seq, int M, int D,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias,
                                                        float eps, float* __restrict__ copy_f32,
                                                        TOut* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const long m = static_cast<long>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  const long slot = m / per_slot;
  const long tok = idx ? static_cast<long>(idx[m]) : (m - slot * per_slot);
  const TIn* row = src + (slot * seq + tok) * D;
  const int groups = D / 8;
  float v[G][8], wv[G][8], bv[G][8];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int g = lane + 64 * i;
    if (g < groups) load8<TIn>(row + g * 8, v[i]);
  }
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int g = lane + 64 * i;
    if (g < groups) {
      load8<float>(w + g * 8, wv[i]);
      load8<float>(bias + g * 8, bv[i]);
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int g = lane + 64 * i;
    if (g < groups) {
#pragma unroll
      for (int j = 0; j < 8; ++j) sum += v[i][j];
    }
  }
  const float inv_d = 1.0f / static_cast<float>(D);
  const float mean = wave_sum(sum) * inv_d;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int g = lane + 64 * i;
    if (g < groups) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[i][j] - mean;
        sq += d * d;
      }
    }
  }
  const float var = wave_sum(sq) * inv_d;
  const float rstd = __builtin_amdgcn_rsqf(var + eps);  // hardware 1/sqrt (about 1 ulp)
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int g = lane + 64 * i;
    if (g < groups) {
      if (copy_f32) store8<float>(copy_f32 + m * D + g * 8, v[i]);
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (v[i][j] - mean) * rstd * wv[i][j] + bv[i][j];
      store8<TOut>(out + m * D + g * 8, o);
    }
  }
}

template <typename TIn, typename TOut, int G>
static hipError_t ln_launch_g(const void* src, const int32_t* idx, int per_slot, int seq, int M,
                              int D, const float* w, const float* b, float eps, float* copy_f32,
                              void* out, hipStream_t st) {
  dim3 grid(static_cast<unsigned>((M + 3) / 4));
  hipLaunchKernelGGL((layernorm_kernel<TIn, TOut, G>), grid, dim3(256), 0, st,
                     static_cast<const TIn*>(src), idx, per_slot, seq, M, D, w, b, eps,
                     copy_f32, static_cast<TOut*>(out));
  return hipGetLastError();
}

template <typename TIn, typename TOut>
static hipError_t ln_launch(const void* src, const int32_t* idx, int per_slot, int seq, int M,
                            int D, const float* w, const float* b, float eps, float* copy_f32,
                            void* out, hipStream_t st) {
  switch ((D / 8 + 63) / 64) {
    case 1: return ln_launch_g<TIn, TOut, 1>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
    case 2: return ln_launch_g<TIn, TOut, 2>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
    case 3: return ln_launch_g<TIn, TOut, 3>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
    case 4: return ln_launch_g<TIn, TOut, 4>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_layernorm(int dtype, const void* src, bool src_f32, const int32_t* idx,
                            int per_slot, int seq, int M, int D, const float* w, const float* b,
                            float eps, float* copy_f32, void* out, hipStream_t st) {
  if (M == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    if (src_f32)
      return ln_launch<float, bf16_t>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
    return ln_launch<bf16_t, bf16_t>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
  }
  return ln_launch<float, float>(src, idx, per_slot, seq, M, D, w, b, eps, copy_f32, out, st);
}

}  // namespace marcache
