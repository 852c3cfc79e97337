// Bidirectional attention of a set of query rows against every key of the
// slot (Eq. 3, no mask): dense for the always-computed blocks (every token
// is a query) and partial for the cached blocks (the N selected rows are the
// queries, keys/values of every token come from the per-block cache).
//
// bf16 path: one workgroup per (slot, head, 64 queries); keys/values stream
// through LDS in blocks of 64 keys with an online softmax, so any sequence
// length works.  The products are the transposed ones (S^T = K Q^T,
// O^T = V^T P^T) so that every query stays in one MFMA column: a lane then
// owns a query's softmax statistics and output, and the probabilities feed
// the second product from the registers that produced them.  The sum over
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

// bf16: WAVES waves of 32 queries per workgroup; keys and values (both
// [key][d] per slot and head) stream through LDS in blocks of 64 keys.
// Per block and wave, with 32x32x16 MFMAs:
//   S^T (32 keys x 32 queries) = K Q^T   A = K rows from LDS, B = Q (registers)
//   O^T (32 d x 32 queries)   += V^T P^T A = V^T fragments, B = P (registers)
// Lane (q, h) = (lane % 32, lane / 32) owns query q: S^T gives it keys
// 8 j + 4 h + i (j, i = 0..3) of each 32-key half, which are exactly the
// eight k-slots it feeds to the second product for each 16-key step (in a
// permuted key order that the V^T operand follows), and O^T gives it rows
// d = 8 j + 4 h + i of its query's output.  The softmax statistics of a
// query live in its two lanes (q and q + 32).
//
// The V^T operand is read from the value rows with ds_read_b64_tr_b16: in
// each group of 16 lanes, lane i receives element i % 4 of the 8 bytes
// addressed by lane 4 s + i / 4, for s = 0..3.  When the group's lanes
// address 4 key rows x 16 columns (lane j: key row j / 4, columns
// 4 (j % 4) .. + 3), lane i therefore receives column i of 4 consecutive
// keys: the 4 keys of one k-slot run of its V^T row.
template <int DH>
constexpr int value_row_stride() {
  // padded d range of the O^T tiles, plus a row offset of 64 bytes modulo
  // 256 so that the four key rows of a transposed read fall on different
  // banks
  int v = (DH + 31) / 32 * 32;
  while ((v * 2) % 256 != 64 && (v * 2) % 256 != 192) v += 8;
  return v;
}

template <int DH, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void attn_bf16_kernel(const bf16_t* __restrict__ Q,
                                                               const bf16_t* __restrict__ Kc,
                                                               const bf16_t* __restrict__ Vc,
                                                               bf16_t* __restrict__ O, int H, int seq,
                                                               int per_slot, float scale_log2) {
  constexpr int KB = 64;               // keys per LDS block
  constexpr int DS = DH / 16;          // k-steps of S^T
  constexpr int DT = (DH + 31) / 32;   // 32-row tiles of O^T
  constexpr int DHP = DT * 32;         // O^T rows incl. padding
  constexpr int KROW = DH + 8;         // key row stride (elements)
  constexpr int VROW = value_row_stride<DH>();  // value row stride (elements), >= DHP
  constexpr int THREADS = 64 * WAVES;
  constexpr int QB = 32 * WAVES;
  __shared__ __align__(16) bf16_t Ks[KB * KROW];
  __shared__ __align__(16) bf16_t Vs[KB * VROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qblocks = (per_slot + QB - 1) / QB;
  const int qb = blockIdx.x % qblocks;
  const int bh = blockIdx.x / qblocks;
  const int h = bh % H;
  const int b = bh / H;
  const int D = H * DH;
  const int ql = lane & 31;
  const int hg = lane >> 5;
  const int qi = qb * QB + wave * 32 + ql;
  const bool q_ok = qi < per_slot;
  const long q_row = static_cast<long>(b) * per_slot + qi;

  u32x4_t qf[DS];  // Q[q][16 s + 8 hg .. + 7]
#pragma unroll
  for (int st = 0; st < DS; ++st)
    qf[st] = q_ok ? *reinterpret_cast<const u32x4_t*>(Q + q_row * D + h * DH + 16 * st + 8 * hg)
                  : u32x4_t{0u, 0u, 0u, 0u};
  if constexpr (DHP > DH) {
    // the d columns past DH feed only O^T rows that are never stored; they
    // are zeroed once so that those rows stay finite
    for (int i = tid; i < KB * (DHP - DH); i += THREADS)
      Vs[(i / (DHP - DH)) * VROW + DH + i % (DHP - DH)] = 0;
  }

  const long head_off = (static_cast<long>(b) * H + h) * seq * DH;
  const bf16_t* kbase = Kc + head_off;
  const bf16_t* vbase = Vc + head_off;
  f32x16_t oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.f;
  float m_run = -__builtin_huge_valf();
  float l_run = 0.f;  // this lane's share of the row sum

  // A block is KB rows of keys and KB rows of values, DH / 8 chunks of 16
  // bytes each, PER_T chunks of each per thread.  The next block is loaded
  // into registers while the current one is multiplied.
  constexpr int CH = DH / 8;
  constexpr int NCHUNK = KB * CH;
  constexpr int PER_T = (NCHUNK + THREADS - 1) / THREADS;
  u32x4_t rk[PER_T], rv[PER_T];
  auto load_block = [&](int key0) {
    if (key0 + KB <= seq) {  // a whole block: no bounds to check
#pragma unroll
      for (int i = 0; i < PER_T; ++i) {
        const int v = min(tid + THREADS * i, NCHUNK - 1);  // a spare thread repeats the last chunk
        const long off = static_cast<long>(key0 + v / CH) * DH + 8 * (v % CH);
        rk[i] = *reinterpret_cast<const u32x4_t*>(kbase + off);
        rv[i] = *reinterpret_cast<const u32x4_t*>(vbase + off);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int v = min(tid + THREADS * i, NCHUNK - 1);
      const int key = key0 + v / CH;
      const long off = static_cast<long>(key) * DH + 8 * (v % CH);
      rk[i] = key < seq ? *reinterpret_cast<const u32x4_t*>(kbase + off) : u32x4_t{0u, 0u, 0u, 0u};
      rv[i] = key < seq ? *reinterpret_cast<const u32x4_t*>(vbase + off) : u32x4_t{0u, 0u, 0u, 0u};
    }
  };
  auto store_block = [&]() {
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int v = tid + THREADS * i;
      if (NCHUNK % THREADS != 0 && v >= NCHUNK) break;
      const int r = v / CH, c = v - (v / CH) * CH;
      *reinterpret_cast<u32x4_t*>(Ks + r * KROW + 8 * c) = rk[i];
      *reinterpret_cast<u32x4_t*>(Vs + r * VROW + 8 * c) = rv[i];
    }
  };
  // transposed reads: key row and d column this lane addresses
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  typedef __attribute__((ext_vector_type(4))) short s16x4_t;
  auto read_tr = [](const bf16_t* p) {
    const s16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_t*)(p));
    return __builtin_bit_cast(u32x2_t, v);
  };

  const int n_blocks = (seq + KB - 1) / KB;
  load_block(0);
  for (int kb = 0; kb < n_blocks; ++kb) {
    const int key0 = kb * KB;
    __syncthreads();  // the previous block is consumed
    store_block();
    __syncthreads();
    if (kb + 1 < n_blocks) load_block(key0 + KB);

    // All K fragments of the block first, then the S^T products, then the
    // V^T fragments of the second product, so that their LDS latency hides
    // under the softmax arithmetic (left alone, the scheduler sinks every
    // read next to its MFMA and each MFMA waits on it).
    u32x4_t kf[2][DS];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int st = 0; st < DS; ++st)
        kf[sb][st] = *reinterpret_cast<const u32x4_t*>(Ks + (32 * sb + ql) * KROW + 16 * st + 8 * hg);
    __builtin_amdgcn_sched_barrier(0);
    f32x16_t sc[2];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[sb][r] = 0.f;
#pragma unroll
      for (int st = 0; st < DS; ++st)
        sc[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf[sb][st]),
                                                         __builtin_bit_cast(bf16x8_t, qf[st]), sc[sb], 0, 0, 0);
    }
    u32x4_t vfr[2][2][DT];  // keys 32 sb + 16 s2 + ..., rows 32 t + ql of V^T
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int t = 0; t < DT; ++t) {
          const bf16_t* vr = Vs + (32 * sb + 16 * s2 + 4 * hg + tr_row) * VROW + 32 * t + tr_col;
          const u32x2_t lo = read_tr(vr);             // keys 4 hg + 0..3 of the 16-key step
          const u32x2_t hi = read_tr(vr + 8 * VROW);  // keys 8 + 4 hg + 0..3
          vfr[sb][s2][t] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
        }
    __builtin_amdgcn_sched_barrier(0);
    // block max of this query over its two lanes, on the unscaled scores
    // (the scale is positive); keys past the end only in a partial block
    float tmax = -__builtin_huge_valf();
    if (key0 + KB <= seq) {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sc[sb][r]);
    } else {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * sb + 8 * (r >> 2) + 4 * hg + (r & 3);
          sc[sb][r] = key < seq ? sc[sb][r] : -__builtin_huge_valf();
          tmax = fmaxf(tmax, sc[sb][r]);
        }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    // Exponents in log2 units against a reference m_run: p = 2^(s scale - m_run).
    // The softmax is the same for any reference, so a query's m_run only
    // moves when its block maximum exceeds it by more than 2^8 (p then stays
    // below 256, far inside the range of bf16 and fp32).  The decision is
    // the query's own; the rescale runs when any query of the wave moves,
    // the others multiplying by exactly 1, so a query's result never
    // depends on which queries share its wave.
    const float m_blk = tmax * scale_log2;
    const bool grow = m_blk > m_run + 8.f;  // always on the first block
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_blk) : 1.f;  // 0 on the first block
      m_run = grow ? m_blk : m_run;
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;
    }
    // the hardware exp2 (no denormal handling: such p are far below what
    // bf16 probabilities can hold next to the block's largest, which is >= 2^-8)
    float psum = 0.f;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[sb][r], scale_log2, -m_run));
        sc[sb][r] = p;
        psum += p;
      }
    l_run += psum;

#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        u32x4_t pf;  // keys 32 sb + 16 s2 + {4 hg + i, 8 + 4 hg + i}
        pf[0] = pack2bf(sc[sb][8 * s2 + 0], sc[sb][8 * s2 + 1]);
        pf[1] = pack2bf(sc[sb][8 * s2 + 2], sc[sb][8 * s2 + 3]);
        pf[2] = pack2bf(sc[sb][8 * s2 + 4], sc[sb][8 * s2 + 5]);
        pf[3] = pack2bf(sc[sb][8 * s2 + 6], sc[sb][8 * s2 + 7]);
#pragma unroll
        for (int t = 0; t < DT; ++t) {
          oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vfr[sb][s2][t]),
                                                            __builtin_bit_cast(bf16x8_t, pf), oacc[t], 0, 0, 0);
        }
      }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!q_ok) return;
  const float inv = 1.0f / l_tot;
  // oacc[t][4 j + i] = O[query][d = 32 t + 8 j + 4 hg + i]
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int d0 = 32 * t + 8 * j + 4 * hg;
      if (d0 < DH) {
        u32x2_t w;
        w[0] = pack2bf(oacc[t][4 * j] * inv, oacc[t][4 * j + 1] * inv);
        w[1] = pack2bf(oacc[t][4 * j + 2] * inv, oacc[t][4 * j + 3] * inv);
        *reinterpret_cast<u32x2_t*>(O + q_row * D + h * DH + d0) = w;
      }
    }
}

// fp32: 64 queries per workgroup, one per lane; keys and values (the
// values transposed on the way in) tiled in LDS.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ Q,
                                                      const float* __restrict__ Kc,
                                                      const float* __restrict__ Vc,
                                                      float* __restrict__ O, int H, int seq,
                                                      int per_slot, float scale_log2) {
  __shared__ float Ks[kKeyTile * DH];
  __shared__ float Vt[DH * kKeyTile];
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
  const float* vbase = Vc + (static_cast<long>(b) * H + h) * seq * DH;  // [seq][DH]
  float m_run = -__builtin_huge_valf(), l_run = 0.f;
  for (int key0 = 0; key0 < seq; key0 += kKeyTile) {
    const int nk = min(kKeyTile, seq - key0);
    __syncthreads();
    for (int e = lane; e < nk * DH; e += 64) Ks[e] = kbase[static_cast<long>(key0) * DH + e];
    for (int e = lane; e < DH * kKeyTile; e += 64) {
      const int d = e / kKeyTile, j = e - d * kKeyTile;
      Vt[e] = j < nk ? vbase[static_cast<long>(key0 + j) * DH + d] : 0.f;
    }
    __syncthreads();
    for (int j = 0; j < nk; ++j) {
      float sdot = 0.f;
#pragma unroll
      for (int d = 0; d < DH; ++d) sdot = fmaf(q[d], Ks[j * DH + d], sdot);
      sdot *= scale_log2;
      const float m_new = fmaxf(m_run, sdot);
      const float alpha = exp2f(m_run - m_new);
      const float p = exp2f(sdot - m_new);
      m_run = m_new;
      l_run = l_run * alpha + p;
#pragma unroll
      for (int d = 0; d < DH; ++d) acc[d] = fmaf(p, Vt[d * kKeyTile + j], acc[d] * alpha);
    }
  }
  if (!q_ok) return;
  const float inv = 1.0f / l_run;
#pragma unroll
  for (int d = 0; d < DH; ++d) O[q_row * D + h * DH + d] = acc[d] * inv;
}

template <int DH, int WAVES>
static void attn_bf16_launch(const void* q, const void* k, const void* v, void* out, int n_slots, int H,
                             int seq, int per_slot, float scale_log2, hipStream_t st) {
  const int qblocks = (per_slot + 32 * WAVES - 1) / (32 * WAVES);
  const long grid = static_cast<long>(n_slots) * H * qblocks;
  hipLaunchKernelGGL((attn_bf16_kernel<DH, WAVES>), dim3(static_cast<unsigned>(grid)), dim3(64 * WAVES), 0, st,
                     static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k), static_cast<const bf16_t*>(v),
                     static_cast<bf16_t*>(out), H, seq, per_slot, scale_log2);
}

template <int DH>
static hipError_t attn_launch(int dtype, const void* q, const void* k, const void* v, void* out,
                              int n_slots, int H, int seq, int per_slot, hipStream_t st) {
  const float scale_log2 = kLog2e / sqrtf(static_cast<float>(DH));
  if (dtype == DT_BF16) {
    // 128 queries per workgroup share each key/value block four ways and,
    // with half the prefetch registers per thread, fit three waves per SIMD
    // for d_head <= 64; below 128 queries per slot the empty query rows of
    // such a workgroup cost more (measured on MI355X: dense MAR-L -17 %,
    // 50-query launches +18 %, d_head 80 +8 %)
    if (per_slot >= 128 && DH <= 64)
      attn_bf16_launch<DH, 4>(q, k, v, out, n_slots, H, seq, per_slot, scale_log2, st);
    else
      attn_bf16_launch<DH, 2>(q, k, v, out, n_slots, H, seq, per_slot, scale_log2, st);
  } else {
    const int qblocks = (per_slot + 63) / 64;
    const long grid = static_cast<long>(n_slots) * H * qblocks;
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
