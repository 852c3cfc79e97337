// Token scoring and selection (Sec. 3.2, Eq. 8).
//
// score: S(x_i) = <v_i, r_i> / (||v_i|| ||r_i||) between this step's value
//   row v_i and the previous step's r_i.  One wave per token; the D = H * dh
//   elements of a row are spread over the heads of the [slot, head, token,
//   dh] cache layout, each lane reads 16-byte chunks.  The products of
//   stored bf16/fp32 values are exact in fp64; each lane keeps an unevaluated
//   sum hi + lo of them (Knuth's two-sum moves every rounding error of hi
//   into lo), the wave combines the pairs the same way, and hi + lo is
//   rounded once.  The three dot products are therefore the exactly rounded
//   sums whatever the lane/summation order (unless the errors themselves
//   span more than 53 bits).  Zero norms give 1 (both rows zero) or 0.  The
//   wave then overwrites r_i with v_i, so the reference always holds the
//   last step's rows.
// select: per slot, the n tokens with the smallest score (NaN ranks as +inf,
//   ties to the lower index), written in ascending token order.  A token's
//   rank is the number of tokens before it in the strict total order
//   (score, index); ranks are a permutation, so exactly n tokens are chosen.
//   The opposite rule (the n largest scores: Table 3's strategy that caches
//   the least similar tokens) ranks by (-score, index), NaN again last.
#include "common.h"

namespace marcache {

// Unevaluated fp64 sum hi + lo.
struct Sum2 {
  double hi, lo;
};

// hi + p = s + e exactly (two-sum, no assumption on magnitudes).
__device__ __forceinline__ void add2(Sum2& a, double p) {
  const double s = a.hi + p;
  const double bb = s - a.hi;
  const double e = (a.hi - (s - bb)) + (p - bb);
  a.hi = s;
  a.lo += e;
}

__device__ __forceinline__ double wave_sum2(Sum2 a) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double oh = __shfl_xor(a.hi, o, 64);
    const double ol = __shfl_xor(a.lo, o, 64);
    a.lo += ol;
    add2(a, oh);
  }
  return a.hi + a.lo;
}

template <typename T>
__global__ __launch_bounds__(256) void scores_kernel(const T* __restrict__ v_cur,
                                                     T* __restrict__ v_ref, int n_slots,
                                                     int H, int seq, int dh,
                                                     double* __restrict__ scores,
                                                     int update_ref) {
  constexpr int PER = Elem<T>::kPer16B;
  const int lane = threadIdx.x & 63;
  const long token = static_cast<long>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (token >= static_cast<long>(n_slots) * seq) return;
  const int b = static_cast<int>(token / seq);
  const int t = static_cast<int>(token % seq);
  const int D = H * dh;
  const int n_chunks = D / PER;
  Sum2 dot{0.0, 0.0}, nv{0.0, 0.0}, nr{0.0, 0.0};
  for (int c = lane; c < n_chunks; c += 64) {
    const int e = c * PER;
    const int h = e / dh;
    const int d = e - h * dh;
    const long off = ((static_cast<long>(b) * H + h) * seq + t) * dh + d;
    const u32x4_t vv = *reinterpret_cast<const u32x4_t*>(v_cur + off);
    const u32x4_t rr = *reinterpret_cast<const u32x4_t*>(v_ref + off);
    float fv[PER], fr[PER];
    unpack16(vv, fv, static_cast<const T*>(nullptr));
    unpack16(rr, fr, static_cast<const T*>(nullptr));
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const double a = fv[i], r = fr[i];
      add2(dot, a * r);
      add2(nv, a * a);
      add2(nr, r * r);
    }
    if (update_ref) *reinterpret_cast<u32x4_t*>(v_ref + off) = vv;
  }
  const double vr = wave_sum2(dot);
  const double vv = wave_sum2(nv);
  const double rr = wave_sum2(nr);
  if (lane == 0) {
    const double den = sqrt(vv * rr);
    double s;
    if (den == 0.0) {
      s = (vv == 0.0 && rr == 0.0) ? 1.0 : 0.0;
    } else {
      s = vr / den;
    }
    scores[token] = s;
  }
}

// One workgroup of 256 threads per slot; scores staged in LDS.
__global__ __launch_bounds__(256) void select_kernel(const double* __restrict__ scores, int seq,
                                                     int n, int largest, int32_t* __restrict__ idx) {
  extern __shared__ double s_lds[];  // [seq] scores, then [256] int counts
  int* cnt = reinterpret_cast<int*>(s_lds + seq);
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const double* s = scores + static_cast<long>(b) * seq;
  for (int t = tid; t < seq; t += 256) {
    double v = largest ? -s[t] : s[t];
    if (v != v) v = __builtin_huge_val();  // NaN ranks last
    s_lds[t] = v;
  }
  __syncthreads();
  // Each thread owns a contiguous run of tokens so that the ascending
  // output order follows from one exclusive scan of the per-thread counts.
  const int per = (seq + 255) / 256;
  const int t0 = tid * per;
  const int t1 = min(t0 + per, seq);
  unsigned long long mask = 0;  // per <= 16 (seq <= 4096)
  int mine = 0;
  for (int t = t0; t < t1; ++t) {
    const double st = s_lds[t];
    int rank = 0;
    for (int j = 0; j < seq; ++j) {
      const double sj = s_lds[j];
      rank += (sj < st) || (sj == st && j < t);
    }
    if (rank < n) {
      mask |= 1ull << (t - t0);
      ++mine;
    }
  }
  cnt[tid] = mine;
  __syncthreads();
  // exclusive scan of 256 counts (serial per thread over at most 256 values)
  int base = 0;
  for (int j = 0; j < tid; ++j) base += cnt[j];
  int32_t* out = idx + static_cast<long>(b) * n;
  for (int t = t0; t < t1; ++t) {
    if (mask & (1ull << (t - t0))) {
      if (base < n) out[base] = t;  // always true: exactly n ranks are < n
      ++base;
    }
  }
}

hipError_t launch_scores(int dtype, const void* v_cur, void* v_ref, int n_slots, int H, int seq,
                         int dh, double* scores, bool update_ref, hipStream_t st) {
  const long tokens = static_cast<long>(n_slots) * seq;
  if (tokens == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>((tokens + 3) / 4));
  if (dtype == DT_BF16) {
    hipLaunchKernelGGL(scores_kernel<bf16_t>, grid, dim3(256), 0, st,
                       static_cast<const bf16_t*>(v_cur), static_cast<bf16_t*>(v_ref), n_slots,
                       H, seq, dh, scores, update_ref ? 1 : 0);
  } else {
    hipLaunchKernelGGL(scores_kernel<float>, grid, dim3(256), 0, st,
                       static_cast<const float*>(v_cur), static_cast<float*>(v_ref), n_slots, H,
                       seq, dh, scores, update_ref ? 1 : 0);
  }
  return hipGetLastError();
}

hipError_t launch_select(const double* scores, int n_slots, int seq, int n, bool largest, int32_t* idx,
                         hipStream_t st) {
  if (n_slots == 0 || n == 0) return hipSuccess;
  const size_t lds = static_cast<size_t>(seq) * sizeof(double) + 256 * sizeof(int);
  hipLaunchKernelGGL(select_kernel, dim3(n_slots), dim3(256), lds, st, scores, seq, n, largest ? 1 : 0, idx);
  return hipGetLastError();
}

}  // namespace marcache
