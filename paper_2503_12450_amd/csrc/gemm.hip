// Matrix products of the block, C = A W^T with fused epilogues.
//
// A [M, K] (activation rows, dense or compact selected rows) and W [N, K]
// (nn.Linear layout) are both K-contiguous, which is what the MFMA operands
// want: each lane feeds 16 bytes of consecutive k.  Tiles of BM x BN are
// staged through LDS in BK-deep slices with a register prefetch of the next
// slice (double-buffered LDS, one barrier per slice).  Four waves split the
// tile 2 x 2; each wave issues 32x32 MFMAs:
//   bf16: v_mfma_f32_32x32x16_bf16 (one per 16 k)
//   fp32: v_mfma_f32_32x32x2_f32   (four per 8 k)
// Accumulation is fp32.  Every output element sums its k in the same order
// whatever the tile shape, M, or the row's position, so a row of a compact
// (selected-row) product is bitwise equal to the same row of the dense one.
//
// Epilogues (the block's elementwise work rides on the product):
//   BIAS      out = C + b                     (storage dtype)
//   GELU      out = gelu_erf(C + b)           (storage dtype)
//   RESIDUAL  out[row'] = resid + C + b       (fp32; row' may scatter into
//                                              the output cache, Eq. 9)
//   QKV       q rows, and key/value rows written straight into the per-block
//             cache at the row's (slot, token): the cache update of Eq. 9.
#include "common.h"

namespace marcache {

template <typename T> struct Mma;

template <> struct Mma<bf16_t> {
  static constexpr int kBK = 64;  // elements per 128-byte LDS row
  static __device__ __forceinline__ void run(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int kBK = 32;
  static __device__ __forceinline__ void run(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[j]), __uint_as_float(b[j]),
                                                  acc, 0, 0, 0);
  }
};

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752440f));
}

template <typename T>
__device__ __forceinline__ void store_elem(T* p, float v);
template <>
__device__ __forceinline__ void store_elem<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_elem<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

// Epilogue for 4 consecutive rows m0..m0+3 at column n.
template <typename T, int KIND>
__device__ __forceinline__ void epilogue4(const EpiArgs& e, int M, int N, int m0, int n,
                                          const float* v) {
  if (n >= N) return;
  const float bias = e.bias[n];
  if constexpr (KIND == EPI_BIAS || KIND == EPI_GELU) {
    T* out = static_cast<T*>(e.out);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i;
      if (m < M) {
        float x = v[i] + bias;
        if constexpr (KIND == EPI_GELU) x = gelu_erf(x);
        store_elem<T>(out + static_cast<long>(m) * N + n, x);
      }
    }
  } else if constexpr (KIND == EPI_RESIDUAL) {
    float* out = static_cast<float*>(e.out);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i;
      if (m < M) {
        const long src = static_cast<long>(m) * N + n;
        const float x = e.resid[src] + (v[i] + bias);
        if (e.out_idx) {
          const long slot = m / e.per_slot;
          out[(slot * e.seq + e.out_idx[m]) * N + n] = x;
          if (e.resid_copy) e.resid_copy[src] = x;
        } else {
          out[src] = x;
        }
      }
    }
  } else {  // EPI_QKV
    const int ng = n + e.n_offset;
    const int sec = ng / e.d_model;
    const int rem = ng - sec * e.d_model;
    const int head = rem / e.d_head;
    const int d = rem - head * e.d_head;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i;
      if (m < M) {
        const float x = v[i] + bias;
        if (sec == 0) {
          store_elem<T>(static_cast<T*>(e.out) + static_cast<long>(m) * e.d_model + rem, x);
        } else {
          const long slot = m / e.per_slot;
          const long tok = e.idx ? static_cast<long>(e.idx[m]) : (m - slot * e.per_slot);
          const long off = ((slot * e.n_heads + head) * e.seq + tok) * e.d_head + d;
          if (sec == 1) {
            store_elem<T>(static_cast<T*>(e.k_cache) + off, x);
          } else {
            store_elem<T>(static_cast<T*>(e.v_cache) + off, x);
            if (e.v_copy) store_elem<T>(static_cast<T*>(e.v_copy) + off, x);
          }
        }
      }
    }
  }
}

template <typename T, int BM, int BN, int KIND>
__global__ __launch_bounds__(256) void gemm_kernel(const T* __restrict__ A,
                                                   const T* __restrict__ W, int M, int N, int K,
                                                   EpiArgs e) {
  constexpr int BK = Mma<T>::kBK;
  constexpr int PER = Elem<T>::kPer16B;       // elements per 16-byte vector
  constexpr int VROW = BK / PER;              // 16-byte vectors per LDS row (8)
  constexpr int LROW = BK + PER;              // padded LDS row (elements): 144 bytes
  constexpr int WM = BM / 2, WN = BN / 2;     // wave tile
  constexpr int TM = WM / 32, TN = WN / 32;   // MFMA tiles per wave
  constexpr int A_LOADS = BM * VROW / 256;    // 16-byte loads per thread per slice
  constexpr int B_LOADS = BN * VROW / 256;

  extern __shared__ __align__(16) unsigned char smem[];
  T* As = reinterpret_cast<T*>(smem);                    // [2][BM][LROW]
  T* Bs = As + 2 * BM * LROW;                            // [2][BN][LROW]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_n = (N + BN - 1) / BN;
  const int tile_m = blockIdx.x / tiles_n;
  const int tile_n = blockIdx.x - tile_m * tiles_n;
  const int m_base = tile_m * BM;
  const int n_base = tile_n * BN;

  u32x4_t ra[A_LOADS], rb[B_LOADS];
  const u32x4_t zero = {0u, 0u, 0u, 0u};

  auto load_slice = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
      const int v = tid + 256 * i;
      const int r = v / VROW, c = v - r * VROW;
      const int m = m_base + r;
      ra[i] = (m < M) ? *reinterpret_cast<const u32x4_t*>(A + static_cast<long>(m) * K + k0 + c * PER)
                      : zero;
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
      const int v = tid + 256 * i;
      const int r = v / VROW, c = v - r * VROW;
      const int n = n_base + r;
      rb[i] = (n < N) ? *reinterpret_cast<const u32x4_t*>(W + static_cast<long>(n) * K + k0 + c * PER)
                      : zero;
    }
  };
  auto store_slice = [&](int buf) {
    T* as = As + buf * BM * LROW;
    T* bs = Bs + buf * BN * LROW;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
      const int v = tid + 256 * i;
      const int r = v / VROW, c = v - r * VROW;
      *reinterpret_cast<u32x4_t*>(as + r * LROW + c * PER) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
      const int v = tid + 256 * i;
      const int r = v / VROW, c = v - r * VROW;
      *reinterpret_cast<u32x4_t*>(bs + r * LROW + c * PER) = rb[i];
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / BK;
  load_slice(0);
  store_slice(0);
  __syncthreads();

  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * PER;  // element offset of this lane's 16 bytes
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_slice((kt + 1) * BK);
    const T* as = As + buf * BM * LROW + (wm * WM + frag_row) * LROW + frag_k;
    const T* bs = Bs + buf * BN * LROW + (wn * WN + frag_row) * LROW + frag_k;
#pragma unroll
    for (int kk = 0; kk < BK / (2 * PER); ++kk) {
      u32x4_t fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const u32x4_t*>(as + i * 32 * LROW + kk * 2 * PER);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const u32x4_t*>(bs + j * 32 * LROW + kk * 2 * PER);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) Mma<T>::run(acc[i][j], fa[i], fb[j]);
    }
    if (kt + 1 < KT) store_slice(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][4*g + r] holds row 8*g + 4*(lane/32) + r, column lane%32 of
  // the 32x32 tile (i, j).
  const int col = lane & 31;
  const int rq = (lane >> 5) * 4;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v4[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                       acc[i][j][4 * g + 3]};
        const int m0 = m_base + wm * WM + i * 32 + 8 * g + rq;
        const int n = n_base + wn * WN + j * 32 + col;
        epilogue4<T, KIND>(e, M, N, m0, n, v4);
      }
}

template <typename T, int BM, int BN, int KIND>
static hipError_t gemm_launch(const void* A, const void* W, int M, int N, int K,
                              const EpiArgs& e, hipStream_t st) {
  constexpr int BK = Mma<T>::kBK;
  constexpr int LROW = BK + Elem<T>::kPer16B;
  const size_t lds = static_cast<size_t>(2) * (BM + BN) * LROW * sizeof(T);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&gemm_kernel<T, BM, BN, KIND>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, KIND>), dim3(tiles), dim3(256), lds, st,
                     static_cast<const T*>(A), static_cast<const T*>(W), M, N, K, e);
  return hipGetLastError();
}

template <typename T, int KIND>
static hipError_t gemm_pick(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                            hipStream_t st) {
  return gemm_launch<T, 128, 128, KIND>(A, W, M, N, K, e, st);
}

template <typename T>
static hipError_t gemm_kind(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                            hipStream_t st) {
  switch (e.kind) {
    case EPI_BIAS: return gemm_pick<T, EPI_BIAS>(A, W, M, N, K, e, st);
    case EPI_GELU: return gemm_pick<T, EPI_GELU>(A, W, M, N, K, e, st);
    case EPI_RESIDUAL: return gemm_pick<T, EPI_RESIDUAL>(A, W, M, N, K, e, st);
    case EPI_QKV: return gemm_pick<T, EPI_QKV>(A, W, M, N, K, e, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(int dtype, const void* A, const void* W, int M, int N, int K,
                       const EpiArgs& e, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  if (dtype == DT_BF16) return gemm_kind<bf16_t>(A, W, M, N, K, e, st);
  return gemm_kind<float>(A, W, M, N, K, e, st);
}

}  // namespace marcache
