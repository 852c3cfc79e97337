// Classifier-free guidance with the condition cache (Sec. 3.1 Eq. 7,
// Sec. 3.2 Eq. 10), elementwise over fp32 rows, 4 elements per lane.
//   STORE: C = u - c, mix with u
//   REUSE: u_hat = c + C, mix with u_hat
//   guided = fmaf(scale, c - u, u)
#include "common.h"

namespace marcache {

template <int OP>
__global__ __launch_bounds__(256) void cfg_kernel(const float* __restrict__ c,
                                                  const float* __restrict__ u,
                                                  float* __restrict__ stored, float scale,
                                                  float* __restrict__ guided,
                                                  float* __restrict__ u_out, size_t count) {
  const size_t i4 = (static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i4 >= count) return;
  const int n = (count - i4 >= 4) ? 4 : static_cast<int>(count - i4);
  float cv[4], uv[4], gv[4];
  if (n == 4) {
    const f32x4_t c4 = *reinterpret_cast<const f32x4_t*>(c + i4);
    for (int j = 0; j < 4; ++j) cv[j] = c4[j];
    if (OP == 0) {
      const f32x4_t u4 = *reinterpret_cast<const f32x4_t*>(u + i4);
      for (int j = 0; j < 4; ++j) uv[j] = u4[j];
    } else {
      const f32x4_t s4 = *reinterpret_cast<const f32x4_t*>(stored + i4);
      for (int j = 0; j < 4; ++j) uv[j] = cv[j] + s4[j];
    }
  } else {
    for (int j = 0; j < n; ++j) {
      cv[j] = c[i4 + j];
      uv[j] = (OP == 0) ? u[i4 + j] : cv[j] + stored[i4 + j];
    }
  }
  for (int j = 0; j < n; ++j) gv[j] = fmaf(scale, cv[j] - uv[j], uv[j]);
  if (n == 4) {
    *reinterpret_cast<f32x4_t*>(guided + i4) = f32x4_t{gv[0], gv[1], gv[2], gv[3]};
    if (OP == 0)
      *reinterpret_cast<f32x4_t*>(stored + i4) =
          f32x4_t{uv[0] - cv[0], uv[1] - cv[1], uv[2] - cv[2], uv[3] - cv[3]};
    if (u_out) *reinterpret_cast<f32x4_t*>(u_out + i4) = f32x4_t{uv[0], uv[1], uv[2], uv[3]};
  } else {
    for (int j = 0; j < n; ++j) {
      guided[i4 + j] = gv[j];
      if (OP == 0) stored[i4 + j] = uv[j] - cv[j];
      if (u_out) u_out[i4 + j] = uv[j];
    }
  }
}

hipError_t launch_cfg(int op, const float* c, const float* u, float* stored, float scale,
                      float* guided, float* u_out, size_t count, hipStream_t st) {
  if (count == 0) return hipSuccess;
  const size_t threads = (count + 3) / 4;
  dim3 grid(static_cast<unsigned>((threads + 255) / 256));
  if (op == 0)
    hipLaunchKernelGGL(cfg_kernel<0>, grid, dim3(256), 0, st, c, u, stored, scale, guided, u_out,
                       count);
  else
    hipLaunchKernelGGL(cfg_kernel<1>, grid, dim3(256), 0, st, c, u, stored, scale, guided, u_out,
                       count);
  return hipGetLastError();
}

}  // namespace marcache
