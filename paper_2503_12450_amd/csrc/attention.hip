// Bidirectional attention of a set of query rows against every key of the
// slot (Eq. 3, no mask): dense for the always-computed blocks (every token
// is a query) and partial for the cached blocks (the N selected rows are the
// queries, keys/values of every token come from the per-block cache).
//
// bf16 path, one workgroup per (slot, head, 64 queries), 16 queries per
// wave.  Keys/values stream through LDS in tiles of 64 keys with an online
// softmax, so any sequence length works.  With 16x16x32 bf16 MFMAs:
//   S^T (keys x queries) = K Q^T          A = K tile rows, B = this wave's Q
//   O^T (d x queries)   += V^T P^T        A = V tile read transposed from
//                                         LDS, B = P straight from the
//                                         registers that produced S^T
// Computing the transposed products keeps every query in one column, so a
// lane owns a query's softmax statistics and its output column; the sum over
// keys in the second product visits each lane's keys in a permuted order,
// which only relabels the reduction index.  A query's result depends only on
// its own row and the slot's keys/values, so a query computed in a partial
// launch is bitwise equal to the same query in a dense launch.
//
// fp32 path: one lane per query with scalar fp32 arithmetic.
#include "common.h"

namespace marcache {

constexpr int kKeyTile = 64;
constexpr float kLog2e = 1.4426950408889634f;

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ Kc,
                                                        const bf16_t* __restrict__ Vc,
                                                        bf16_t* __restrict__ O, int H, int seq,
                                                        int per_slot, float scale_log2) {
  constexpr int DC = (DH + 31) / 32;   // 32-wide d chunks of the first product
  constexpr int DT = DH / 16;          // 16-wide d tiles of the output
  constexpr int KROW = DH + 8;         // padded K row (elements)
  constexpr int VROW = kKeyTile + 8;   // padded V^T row (elements)
  __shared__ __align__(16) bf16_t Ks[kKeyTile * KROW];
  __shared__ __align__(16) bf16_t Vt[DH * VROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qblocks = (per_slot + 63) / 64;
  const int qb = blockIdx.x % qblocks;
  const int bh = blockIdx.x / qblocks;
  const int h = bh % H;
  const int b = bh / H;
  const int D = H * DH;

  const int ql = lane & 15;   // this lane's query within the wave
  const int g = lane >> 4;    // lane group 0..3
  const int qi = qb * 64 + wave * 16 + ql;
  const bool q_ok = qi < per_slot;
  const long q_row = static_cast<long>(b) * per_slot + qi;

  // B operand of S^T = K Q^T: Q[q][32 c + 8 g .. + 7]
  u32x4_t qf[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) {
    const int d0 = 32 * c + 8 * g;
    if (q_ok && d0 < DH)
      qf[c] = *reinterpret_cast<const u32x4_t*>(Q + q_row * D + h * DH + d0);
    else
      qf[c] = u32x4_t{0u, 0u, 0u, 0u};
  }

  const bf16_t* kbase = Kc + (static_cast<long>(b) * H + h) * seq * DH;
  const bf16_t* vbase = Vc + (static_cast<long>(b) * H + h) * seq * DH;

  f32x4_t oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) oacc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_huge_valf();
  float l_run = 0.f;  // this lane's share of the row sum

  constexpr int VEC_PER_ROW = DH / 8;
  constexpr int TILE_VECS = kKeyTile * VEC_PER_ROW;
  const int n_tiles = (seq + kKeyTile - 1) / kKeyTile;
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int key0 = kt * kKeyTile;
    __syncthreads();  // previous tile fully consumed
    for (int v = tid; v < TILE_VECS; v += 256) {
      const int r = v / VEC_PER_ROW;
      const int c = v - r * VEC_PER_ROW;
      const int key = key0 + r;
      u32x4_t kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
      if (key < seq) {
        kv = *reinterpret_cast<const u32x4_t*>(kbase + static_cast<long>(key) * DH + c * 8);
        vv = *reinterpret_cast<const u32x4_t*>(vbase + static_cast<long>(key) * DH + c * 8);
      }
      *reinterpret_cast<u32x4_t*>(Ks + r * KROW + c * 8) = kv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        Vt[(c * 8 + 2 * i) * VROW + r] = static_cast<bf16_t>(vv[i] & 0xFFFFu);
        Vt[(c * 8 + 2 * i + 1) * VROW + r] = static_cast<bf16_t>(vv[i] >> 16);
      }
    }
    __syncthreads();

    // S^T for 4 subtiles of 16 keys: s[j][i] = key 16 j + 4 g + i, query ql
    f32x4_t s[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      s[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < DC; ++c) {
        const int d0 = 32 * c + 8 * g;
        u32x4_t kf = {0u, 0u, 0u, 0u};
        if (d0 < DH) kf = *reinterpret_cast<const u32x4_t*>(Ks + (16 * j + ql) * KROW + d0);
        s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                       __builtin_bit_cast(bf16x8_t, qf[c]),
                                                       s[j], 0, 0, 0);
      }
    }
    // scale, mask, tile max of this query across its four lanes
    float tmax = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = key0 + 16 * j + 4 * g + i;
        const float x = (key < seq) ? s[j][i] * scale_log2 : -__builtin_huge_valf();
        s[j][i] = x;
        tmax = fmaxf(tmax, x);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = exp2f(s[j][i] - m_new);
        s[j][i] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) oacc[t][i] *= alpha;

    // O^T += V^T P^T over two 32-key chunks; this lane's k-slots are keys
    // {32 c + 4 g + i} and {32 c + 16 + 4 g + i}, i = 0..3
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      u32x4_t pf;
      pf[0] = pack2bf(s[2 * c][0], s[2 * c][1]);
      pf[1] = pack2bf(s[2 * c][2], s[2 * c][3]);
      pf[2] = pack2bf(s[2 * c + 1][0], s[2 * c + 1][1]);
      pf[3] = pack2bf(s[2 * c + 1][2], s[2 * c + 1][3]);
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const bf16_t* vr = Vt + (16 * t + ql) * VROW + 32 * c + 4 * g;
        const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vr);
        const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vr + 16);
        const u32x4_t vf = {lo[0], lo[1], hi[0], hi[1]};
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vf),
                                                          __builtin_bit_cast(bf16x8_t, pf),
                                                          oacc[t], 0, 0, 0);
      }
    }
  }

  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (!q_ok) return;
  const float inv = 1.0f / l_tot;
  // oacc[t][i] = O[query ql][d = 16 t + 4 g + i]
#pragma unroll
  for (int t = 0; t < DT; ++t) {
    u32x2_t w;
    w[0] = pack2bf(oacc[t][0] * inv, oacc[t][1] * inv);
    w[1] = pack2bf(oacc[t][2] * inv, oacc[t][3] * inv);
    *reinterpret_cast<u32x2_t*>(O + q_row * D + h * DH + 16 * t + 4 * g) = w;
  }
}

// fp32: 64 queries per workgroup, one per lane; keys/values tiled in LDS.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ Q,
                                                      const float* __restrict__ Kc,
                                                      const float* __restrict__ Vc,
                                                      float* __restrict__ O, int H, int seq,
                                                      int per_slot, float scale_log2) {
  __shared__ float Ks[kKeyTile * DH];
  __shared__ float Vs[kKeyTile * DH];
  const int lane = threadIdx.x;
  const int qblocks = (per_slot + 63) / 64;
  const int qb = blockIdx.x % qblocks;
  const int bh = blockIdx.x / qblocks;
  const int h = bh % H;
  const int b = bh / H;
  const int D = H * DH;
  const int qi = qb * 64 + lane;
  const bool q_ok = qi < per_slot;
  const long q_row = static_cast<long>(b) * per_slot + qi;
  float q[DH], acc[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    q[d] = q_ok ? Q[q_row * D + h * DH + d] : 0.f;
    acc[d] = 0.f;
  }
  const float* kbase = Kc + (static_cast<long>(b) * H + h) * seq * DH;
  const float* vbase = Vc + (static_cast<long>(b) * H + h) * seq * DH;
  float m_run = -__builtin_huge_valf(), l_run = 0.f;
  for (int key0 = 0; key0 < seq; key0 += kKeyTile) {
    const int nk = min(kKeyTile, seq - key0);
    __syncthreads();
    for (int e = lane; e < nk * DH; e += 64) {
      Ks[e] = kbase[static_cast<long>(key0) * DH + e];
      Vs[e] = vbase[static_cast<long>(key0) * DH + e];
    }
    __syncthreads();
    for (int j = 0; j < nk; ++j) {
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < DH; ++d) s = fmaf(q[d], Ks[j * DH + d], s);
      s *= scale_log2;
      const float m_new = fmaxf(m_run, s);
      const float alpha = exp2f(m_run - m_new);
      const float p = exp2f(s - m_new);
      m_run = m_new;
      l_run = l_run * alpha + p;
#pragma unroll
      for (int d = 0; d < DH; ++d) acc[d] = fmaf(p, Vs[j * DH + d], acc[d] * alpha);
    }
  }
  if (!q_ok) return;
  const float inv = 1.0f / l_run;
#pragma unroll
  for (int d = 0; d < DH; ++d) O[q_row * D + h * DH + d] = acc[d] * inv;
}

template <int DH>
static hipError_t attn_launch(int dtype, const void* q, const void* k, const void* v, void* out,
                              int n_slots, int H, int seq, int per_slot, hipStream_t st) {
  const int qblocks = (per_slot + 63) / 64;
  const long grid = static_cast<long>(n_slots) * H * qblocks;
  const float scale_log2 = kLog2e / sqrtf(static_cast<float>(DH));
  if (dtype == DT_BF16) {
    hipLaunchKernelGGL(attn_bf16_kernel<DH>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, st,
                       static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                       static_cast<const bf16_t*>(v), static_cast<bf16_t*>(out), H, seq,
                       per_slot, scale_log2);
  } else {
    hipLaunchKernelGGL(attn_f32_kernel<DH>, dim3(static_cast<unsigned>(grid)), dim3(64), 0, st,
                       static_cast<const float*>(q), static_cast<const float*>(k),
                       static_cast<const float*>(v), static_cast<float*>(out), H, seq, per_slot,
                       scale_log2);
  }
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v, void* out,
                            int n_slots, int H, int seq, int dh, int per_slot, hipStream_t st) {
  if (n_slots == 0 || per_slot == 0) return hipSuccess;
  switch (dh) {
    case 16: return attn_launch<16>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 32: return attn_launch<32>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 48: return attn_launch<48>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 64: return attn_launch<64>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 80: return attn_launch<80>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 96: return attn_launch<96>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 112: return attn_launch<112>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    case 128: return attn_launch<128>(dtype, q, k, v, out, n_slots, H, seq, per_slot, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace marcache
