// Matrix products of the block, C = A W^T with fused epilogues.
//
// A [M, K] (activation rows, dense or compact selected rows) and W [N, K]
// (nn.Linear layout) are both K-contiguous, which is what the MFMA operands
// want: each lane feeds 16 bytes of consecutive k.
//
// Data movement: each workgroup owns a BM x BN output tile and walks K in
// slices of 128 bytes per row.  Slices are copied from HBM/L2 straight into
// LDS by buffer loads with the LDS destination (no register staging), into
// a ring of STAGES buffers: slice kt+STAGES-1 is in flight while slice kt is
// multiplied.  Buffer descriptors cover only the tile's rows, so rows past M
// (N) read as zeros without any masking.  Within a 128-byte row the eight
// 16-byte chunks are XOR-swizzled by (row / 2) % 8, which spreads the 16
// lanes of each LDS read phase over all 64 banks.
//
// Math: 32x32 MFMA tiles per wave,
//   bf16: v_mfma_f32_32x32x16_bf16 (one per 16 k)
//   fp32: v_mfma_f32_32x32x2_f32   (four per 8 k)
// with fp32 accumulation; each tile is formed transposed (weights as the
// first operand) so that a lane ends up holding a run of one row.  Every output element sums its k in the same order
// whatever the tile shape, M, or the row's position, so a row of a compact
// (selected-row) product is bitwise equal to the same row of the dense one.
//
// Epilogues (the block's elementwise work rides on the product):
//   BIAS      out = C + b                     (storage dtype)
//   GELU      out = gelu(C + b)               (storage dtype; erf by
//                                              Abramowitz & Stegun 7.1.26 in
//                                              fp32, 7.1.27 for bf16 output)
//   RESIDUAL  out[row'] = resid + C + b       (fp32; row' may scatter into
//                                              the output cache, Eq. 9)
//   SILU      out = silu(C + b)               (bf16)
//   GATE      out = resid + gate (C + b)      (fp32; the gated residual of
//                                              the diffusion head's blocks)
//   QKV       q rows, and keys/values written straight into the per-block
//             cache at the row's (slot, token): the cache update of Eq. 9.
//             Keys and values are both stored [slot, head, token, d]
//             (whole 16-byte row chunks, also for scattered tokens).
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace marcache {

template <typename T> struct Mma;

// One k-step = 32 bytes of K per row (two 16-byte chunks, one per lane half).
template <> struct Mma<bf16_t> {
  static __device__ __forceinline__ void run(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static __device__ __forceinline__ void run(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[j]), __uint_as_float(b[j]),
                                                  acc, 0, 0, 0);
  }
};

// GELU x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)), with erf from Abramowitz &
// Stegun, Handbook of Mathematical Functions, formula 7.1.26:
//   erf(z) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-z^2),
//   t = 1 / (1 + p z), z >= 0, |error| <= 1.5e-7,
// far below the bf16 rounding of the product it feeds.  With
// q = (1 - erf(|x| / sqrt 2)) / 2:  gelu(x) = x (1 - q) for x >= 0, x q else.
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = fabsf(x) * 0.70710678118654752440f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.0f));
  float poly = fmaf(1.061405429f, t, -1.453152027f);
  poly = fmaf(poly, t, 1.421413741f);
  poly = fmaf(poly, t, -0.284496736f);
  poly = fmaf(poly, t, 0.254829592f);
  poly *= t;
  const float q = 0.5f * poly * __expf(-z * z);
  return x >= 0.0f ? x * (1.0f - q) : x * q;
}

// The same GELU for outputs stored in bf16, with erf from Abramowitz &
// Stegun formula 7.1.27:
//   erf(z) = 1 - 1 / (1 + a1 z + a2 z^2 + a3 z^3 + a4 z^4)^4,  z >= 0,
//   |error| <= 5e-4,
// so with z = |x| / sqrt(2), q = (1 - erf(z)) / 2 = 1 / (2^(1/4) D)^4: the
// polynomial is taken in |x| with its coefficients scaled by 2^(1/4) and
// powers of 1/sqrt(2), and one reciprocal gives q.  gelu = x (1 - q) for
// x >= 0 and x q for x < 0, which is max(x, 0) - |x| q for both signs.
// The error in gelu is at most 2.4e-4 |x|, a sixteenth of a bf16 step.
__device__ __forceinline__ float gelu_erf_bf16(float x) {
  const float ax = fabsf(x);
  float d = fmaf(0.0232216473f, ax, 0.000408675658f);  // 2^(1/4) (a4 / 4, a3 / 2^(3/2))
  d = fmaf(d, ax, 0.136990119f);                       // 2^(1/4) a2 / 2
  d = fmaf(d, ax, 0.234099676f);                       // 2^(1/4) a1 / 2^(1/2)
  d = fmaf(d, ax, 1.18920712f);                        // 2^(1/4)
  const float r = __builtin_amdgcn_rcpf(d);
  const float r2 = r * r;
  return fmaf(-(ax * r2), r2, fmaxf(x, 0.0f));
}

// silu(x) = x / (1 + e^-x), with the hardware exp2 and reciprocal (each
// within a few fp32 ulps; the result is stored in bf16).  For x below
// about -88 the exponential overflows to +inf and the quotient is -0,
// the limit.
__device__ __forceinline__ float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

typedef __attribute__((ext_vector_type(4))) int i32x4_t;

// Buffer descriptor over `bytes` bytes at `base` (raw, no stride).
__device__ __forceinline__ i32x4_t make_rsrc(const void* base, unsigned bytes) {
  const unsigned long p = reinterpret_cast<unsigned long>(base);
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(p & 0xFFFFFFFFu));
  r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>(p >> 32));
  r[2] = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
  r[3] = 0x00020000;
  return r;
}

// Sixteen bytes per lane from the buffer (byte offset voff + soff) into LDS at
// lds_addr + 16 * lane.  Issued from asm so the compiler adds no waits of its
// own (it would drain every load before each LDS read); the main loop waits
// with s_waitcnt vmcnt for exactly the slice it is about to read.
// m0 is reserved by the compiler but nothing else in these kernels uses it
// (no LDS-DMA builtins, GWS or messages), so clobbering it here is safe.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(i32x4_t rsrc, unsigned lds_addr, int voff, int soff) {
  // the descriptor is wave-uniform; readfirstlane keeps it in SGPRs even
  // when it was picked by a select (a no-op when it is scalar already)
  i32x4_t r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_readfirstlane(rsrc[i]);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier that waits for this wave's LDS operations only (a
// __syncthreads would also drain the vector-memory counter, i.e. the loads
// already in flight for later slices).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

constexpr int cmin(int a, int b) { return a < b ? a : b; }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
// A wave has at most 63 such operations outstanding (issue stalls at that
// count), so a wait for "all but the last N" with N >= 63 is a wait for all
// but the last 63.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}


// ---------------------------------------------------------------------------
// Epilogues.  The MFMA forms C^T = W A^T (weight fragment as its first
// operand), so that acc[4 g + r] of a lane's 32 x 32 tile is output row
// m_tile + lane % 32 and column n_tile + 8 g + 4 (lane / 32) + r: each lane
// owns one row and four consecutive columns per group g.
//
// A wave finishes its tile one 32-row strip at a time: the strip's values
// (bias added, activation applied, in the output type) are written to a
// private LDS region as row-major rows, then read back as 16-byte chunks so
// that eight consecutive lanes store one whole 128-byte line.  Stores go
// through buffer descriptors; a chunk whose offset falls outside the
// descriptor (rows past M, columns past N, absent outputs of size 0) is
// dropped by the hardware range check, so no store needs a branch.  Offsets
// are 32-bit: the launcher keeps every output below 2 GiB.  N is a multiple
// of 8, so a chunk is wholly inside N or wholly outside.
// ---------------------------------------------------------------------------
constexpr int kOob = 0x7FFFFFF0;  // an offset past every descriptor

typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_out(void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ void bstore16(rsrc_t r, int voff, const u32x4_t& v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, 0, 0);
}
__device__ __forceinline__ u32x4_t bload16(rsrc_t r, int voff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0);
}
__device__ __forceinline__ void bstore1(rsrc_t r, int voff, float x, float*) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, voff, 0, 0);
}
__device__ __forceinline__ void bstore1(rsrc_t r, int voff, float x, bf16_t*) {
  __builtin_amdgcn_raw_buffer_store_b16(f2bf(x), r, voff, 0, 0);
}
// four consecutive output values into LDS
__device__ __forceinline__ void lds_put4(unsigned char* p, const float* x, float*) {
  *reinterpret_cast<f32x4_t*>(p) = f32x4_t{x[0], x[1], x[2], x[3]};
}
__device__ __forceinline__ void lds_put4(unsigned char* p, const float* x, bf16_t*) {
  *reinterpret_cast<u32x2_t*>(p) = u32x2_t{pack2bf(x[0], x[1]), pack2bf(x[2], x[3])};
}

// Descriptors of an epilogue's outputs and inputs.
template <typename T, int KIND>
struct EpiCtx {
  rsrc_t out, aux0, aux1, aux2;
};

template <typename T, int KIND>
__device__ __forceinline__ EpiCtx<T, KIND> make_epi(const EpiArgs& e, int M, int N) {
  constexpr unsigned ES = sizeof(T);
  EpiCtx<T, KIND> c;
  if constexpr (KIND == EPI_BIAS || KIND == EPI_GELU) {
    c.out = make_out(e.out, static_cast<unsigned>(M) * N * ES);
    c.aux0 = c.aux1 = c.aux2 = c.out;
  } else if constexpr (KIND == EPI_SILU) {
    c.out = make_out(e.out, static_cast<unsigned>(M) * N * ES);
    c.aux0 = c.aux1 = c.aux2 = c.out;
  } else if constexpr (KIND == EPI_GATE) {
    c.out = make_out(e.out, static_cast<unsigned>(M) * N * 4u);
    c.aux0 = make_out(const_cast<float*>(e.resid), static_cast<unsigned>(M) * N * 4u);
    c.aux1 = c.aux0;
    c.aux2 = make_out(const_cast<void*>(e.gate), static_cast<unsigned>(M) * e.gate_ld * ES);
  } else if constexpr (KIND == EPI_RESIDUAL) {
    const unsigned rows = e.out_idx ? static_cast<unsigned>((M + e.per_slot - 1) / e.per_slot) * e.seq
                                    : static_cast<unsigned>(M);
    c.out = make_out(e.out, rows * N * 4u);
    c.aux0 = make_out(const_cast<float*>(e.resid), static_cast<unsigned>(M) * N * 4u);
    c.aux1 = make_out(e.resid_copy, e.resid_copy ? static_cast<unsigned>(M) * N * 4u : 0u);
    c.aux2 = c.aux1;
  } else {
    const unsigned slots = static_cast<unsigned>((M + e.per_slot - 1) / e.per_slot);
    const unsigned cache = slots * e.n_heads * e.seq * e.d_head * ES;
    c.out = make_out(e.out, e.out ? static_cast<unsigned>(M) * e.d_model * ES : 0u);
    c.aux0 = make_out(e.k_cache, e.k_cache ? cache : 0u);
    c.aux1 = make_out(e.v_cache, e.v_cache ? cache : 0u);
    c.aux2 = make_out(e.v_copy, e.v_copy ? cache : 0u);
  }
  return c;
}

// QKV column section of global column ng: 0 query, 1 key, 2 value
__device__ __forceinline__ int qkv_section(const EpiArgs& e, int ng) {
  return ng >= 2 * e.d_model ? 2 : (ng >= e.d_model ? 1 : 0);
}

// Epilogue of one 32-row strip of a wave's tile: rows m_strip + 0..31,
// columns n_wave + 0..WN-1; sb is the bias of those columns (LDS), reg the
// wave's LDS staging region (32 * WN * 4 bytes).
template <typename T, int KIND>
using EpiOut = typename std::conditional<KIND == EPI_RESIDUAL || KIND == EPI_GATE, float, T>::type;  // output type

// Rows r0 .. r0 + HS - 1 of the strip go through LDS in one pass (HS = 32,
// or 16 when a 32-row region per wave does not fit the staging space).
template <typename T, int KIND, int WN, int HS>
__device__ __forceinline__ void epilogue_strip(const EpiArgs& e, const EpiCtx<T, KIND>& c, int M, int N,
                                               int m_strip, int n_wave, int lane, const float* sb,
                                               const f32x16_t (&acc)[WN / 32], unsigned char* reg, int r0) {
  constexpr int TN = WN / 32;
  typedef EpiOut<T, KIND> OT;
  constexpr int OS = sizeof(OT);
  constexpr int RB = WN * OS;        // bytes per staged row
  constexpr int NCH = RB / 16;       // 16-byte chunks per row
  constexpr int COLS = 16 / OS;      // columns per chunk
  static_assert((NCH & (NCH - 1)) == 0 && (HS * NCH) % 64 == 0, "chunks per staged row");
  const int row = lane & 31, h4 = (lane >> 5) * 4;
  const int lr = row - r0;  // staged row of this lane, when in [0, HS)
  const bool in_pass = HS == 32 || static_cast<unsigned>(lr) < static_cast<unsigned>(HS);

  // 1. bias (+ activation) in registers, rows into LDS; chunk c of row r sits
  //    at chunk c ^ (r % NCH), which spreads a wave's accesses over the banks
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    float x[4][4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4_t bv = *reinterpret_cast<const f32x4_t*>(sb + 32 * j + 8 * g + h4);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        x[g][r] = acc[j][4 * g + r] + bv[r];
        if constexpr (KIND == EPI_GELU) x[g][r] = sizeof(T) == 2 ? gelu_erf_bf16(x[g][r]) : gelu_erf(x[g][r]);
        if constexpr (KIND == EPI_SILU) x[g][r] = silu_f(x[g][r]);
      }
      const int colb = (32 * j + 8 * g + h4) * OS;
      if (in_pass)
        lds_put4(reg + lr * RB + ((((colb >> 4) ^ lr) & (NCH - 1)) << 4) + (colb & 15), x[g],
                 static_cast<OT*>(nullptr));
    }
  }

  // 2. 16-byte chunks back out of LDS, eight lanes per 128 bytes of a row.
  //    Every load of the pass (LDS chunks, residual rows, row indices) is
  //    issued before any store: an output may alias the residual input, so
  //    the compiler would otherwise keep each load behind the previous
  //    chunk's store and pay a memory round trip per chunk.  Each element is
  //    read before it is written, so the order is safe in place.
  constexpr int IT = HS * NCH / 64;
  u32x4_t val[IT];
  int mrow[IT], ncol[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int v = lane + 64 * it;
    const int r = v / NCH, ch = v & (NCH - 1);
    val[it] = *reinterpret_cast<const u32x4_t*>(reg + r * RB + (((ch ^ r) & (NCH - 1)) << 4));
    mrow[it] = m_strip + r0 + r;
    ncol[it] = n_wave + ch * COLS;
  }
  if constexpr (KIND == EPI_BIAS || KIND == EPI_GELU || KIND == EPI_SILU) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const bool ok = mrow[it] < M && ncol[it] < N;
      bstore16(c.out, ok ? (mrow[it] * N + ncol[it]) * OS : kOob, val[it]);
    }
  } else if constexpr (KIND == EPI_GATE) {
    // y = resid + gate (C + b): four fp32 residual values and four gates
    // (8 bytes of bf16) per chunk, all loaded before the first store
    u32x4_t res[IT];
    u32x2_t gt[IT];
    int lin[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const bool ok = mrow[it] < M && ncol[it] < N;
      const int mc = min(mrow[it], M - 1);
      lin[it] = ok ? (mc * N + ncol[it]) * 4 : kOob;
      res[it] = bload16(c.aux0, lin[it]);
      gt[it] = __builtin_amdgcn_raw_buffer_load_b64(c.aux2, ok ? (mc * e.gate_ld + ncol[it]) * 2 : kOob, 0, 0);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      u32x4_t y;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t gw = gt[it][q >> 1];
        const float g = __uint_as_float((q & 1) ? (gw & 0xFFFF0000u) : (gw << 16));
        y[q] = __float_as_uint(fmaf(g, __uint_as_float(val[it][q]), __uint_as_float(res[it][q])));
      }
      bstore16(c.out, lin[it], y);
    }
  } else if constexpr (KIND == EPI_RESIDUAL) {
    u32x4_t res[IT];
    int lin[IT], orow[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const bool ok = mrow[it] < M && ncol[it] < N;
      const int mc = min(mrow[it], M - 1);
      lin[it] = ok ? (mc * N + ncol[it]) * 4 : kOob;
      res[it] = bload16(c.aux0, lin[it]);
      orow[it] = e.out_idx ? div_by(mc, e.slot_magic, e.slot_shift) * e.seq + e.out_idx[mc] : mc;
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      u32x4_t y;
#pragma unroll
      for (int q = 0; q < 4; ++q) y[q] = __float_as_uint(__uint_as_float(res[it][q]) + __uint_as_float(val[it][q]));
      bstore16(c.out, lin[it] != kOob ? (orow[it] * N + ncol[it]) * 4 : kOob, y);
      if (e.resid_copy) bstore16(c.aux1, lin[it], y);
    }
  } else {
    int tok[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int mc = min(mrow[it], M - 1);
      tok[it] = e.idx ? e.idx[mc] : mc - div_by(mc, e.slot_magic, e.slot_shift) * e.per_slot;
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const bool ok = mrow[it] < M && ncol[it] < N;
      const int mc = min(mrow[it], M - 1);
      const int ng = ncol[it] + e.n_offset;
      const int sec = qkv_section(e, ng);
      const int rem = ng - sec * e.d_model;  // head * d_head + d
      const int slot = div_by(mc, e.slot_magic, e.slot_shift);
      const int head = div_by(rem, e.head_magic, e.head_shift);
      // [slot, head, tok, d]
      const int krow = ((slot * e.n_heads + head) * e.seq + tok[it]) * e.d_head + (rem - head * e.d_head);
      bstore16(c.out, ok && sec == 0 ? (mc * e.d_model + rem) * OS : kOob, val[it]);
      bstore16(c.aux0, ok && sec == 1 ? krow * OS : kOob, val[it]);
      bstore16(c.aux1, ok && sec == 2 ? krow * OS : kOob, val[it]);
      if (e.v_copy) bstore16(c.aux2, ok && sec == 2 ? krow * OS : kOob, val[it]);
    }
  }
}

// Workgroup -> output tile.  Workgroups are dispatched round-robin over the
// eight XCDs (workgroup b runs on XCD b % 8), and each XCD has its own L2.
// Each XCD is given a contiguous range of the tile order, and that order
// walks kGroupM row tiles before moving to the next column tile, so the
// ~32 workgroups an XCD runs at once share 4 row tiles of A and 8 column
// tiles of W instead of touching every row tile of A.  The map is a
// bijection for any tile count.
constexpr int kXcds = 8;
constexpr int kGroupM = 4;
__device__ __forceinline__ void tile_of(int b, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  const int q = total / kXcds, r = total - q * kXcds;
  const int x = b % kXcds, l = b / kXcds;
  const int t = x * q + min(x, r) + l;  // position in the tile order
  const int group = kGroupM * tiles_n;
  const int g = t / group, first_m = g * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int in = t - g * group;
  tm = first_m + in % gm;
  tn = in / gm;
}

// Tile BM x BN, WAVES_M x WAVES_N waves, each wave (BM / WAVES_M) x
// (BN / WAVES_N); STAGES LDS buffers of (BM + BN) rows x ROWB bytes of K.
// Within a row the 16-byte chunks are XOR-swizzled by (row / RPB) % NCH,
// RPB = 256 / ROWB rows per 256 bytes of banks: the 16 lanes of one LDS
// read phase (16 rows, one chunk each) then hit 16 distinct bank groups.
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int ROWB, int KIND, bool PERSIST>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_kernel(const T* __restrict__ A,
                                                                    const T* __restrict__ W, int M,
                                                                    int N, int K, EpiArgs e) {
  constexpr int NW = WAVES_M * WAVES_N;
  // LDS: the A rows of all stages, then the W rows of all stages, so that a
  // fragment's stage and tile offsets fit the 16-bit immediate of ds_read
  constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
  constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  constexpr int B_RING = STAGES * A_BYTES;
  constexpr int NCH = ROWB / 16;               // 16-byte chunks per row
  constexpr int RPB = 256 / ROWB;              // rows per 256 bytes
  constexpr int RPI = 1024 / ROWB;             // rows per wave-wide (1 KiB) load
  constexpr int A_INSTR = BM / RPI / NW;
  constexpr int B_INSTR = BN / RPI / NW;
  constexpr int LOADS = A_INSTR + B_INSTR;     // loads per wave per slice
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int KSTEPS = ROWB / 32;            // MFMA k-steps per slice
  static_assert(ROWB == 64 || ROWB == 128, "slice width");
  static_assert(A_INSTR * RPI * NW == BM && B_INSTR * RPI * NW == BN, "tile/waves");
  static_assert(STAGES >= 2 && STAGES <= 5, "stages");

  __shared__ __align__(1024) unsigned char ring[STAGES * STAGE_BYTES];
  __shared__ __align__(16) float sbias[2][256];  // the bias of the current and the next tile
  static_assert(BN <= 256, "bias slot");
  // Epilogue staging, each wave in its own region of HS rows x WN outputs.
  // One tile per workgroup: the whole ring, once its loads have drained.
  // Persistent: the stage that held the tile's last slice, the one stage
  // not receiving the next tile's first slices (A part first, then W part);
  // HS drops to 16 rows when 32 do not fit.
  typedef EpiOut<T, KIND> OT;
  constexpr int OSZ = static_cast<int>(sizeof(OT));
  constexpr int EC = WN < 64 ? WN : 64;  // columns per epilogue pass
  constexpr int HS = !PERSIST || (A_BYTES / (32 * EC * OSZ)) + (B_BYTES / (32 * EC * OSZ)) >= NW ? 32 : 16;
  constexpr int REGION = HS * EC * OSZ;
  constexpr int REG_IN_A = PERSIST ? A_BYTES / REGION : NW;
  static_assert(PERSIST ? REG_IN_A + B_BYTES / REGION >= NW : NW * REGION <= STAGES * STAGE_BYTES,
                "epilogue staging space");
  // vector-memory operations each wave's epilogue issues whatever the
  // arguments: a store per chunk per output (three for QKV), plus the
  // residual loads.  The optional outputs and the index loads are left out,
  // which only makes the waits that count on this number stricter.
  constexpr int EPI_IT = HS * (EC * OSZ / 16) / 64;
  constexpr int EPI_STRIPS = TM * (TN / (EC / 32)) * (32 / HS);
  constexpr int EPI_OPS = EPI_STRIPS * EPI_IT * (KIND == EPI_RESIDUAL ? 2 : (KIND == EPI_QKV || KIND == EPI_GATE) ? 3 : 1);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave - (wave / WAVES_N) * WAVES_N;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  const int Kb = K * static_cast<int>(sizeof(T));
  const int KT = Kb / ROWB;  // K * sizeof(T) is a multiple of 128

  // operand descriptors of tile t (rows past M / N read as zeros)
  auto tile_rsrc = [&](int t, i32x4_t& ra, i32x4_t& rb, i32x4_t& rbias) {
    int tm, tn;
    tile_of(t, tiles_m, tiles_n, tm, tn);
    ra = make_rsrc(A + static_cast<long>(tm) * BM * K, static_cast<unsigned>(min(BM, M - tm * BM)) * Kb);
    rb = make_rsrc(W + static_cast<long>(tn) * BN * K, static_cast<unsigned>(min(BN, N - tn * BN)) * Kb);
    rbias = make_rsrc(e.bias + tn * BN, static_cast<unsigned>(min(BN, N - tn * BN)) * 4u);
  };

  // A wave-wide load moves RPI rows (group grp) of one slice: lane -> row
  // grp*RPI + r_in, physical chunk pc.  The row's swizzle is
  // (4 grp + r_in / RPB) % NCH, so two lane offsets (even and odd groups)
  // serve every group; the group's row offset is wave-uniform and rides in
  // the scalar offset.
  static_assert(A_INSTR % 2 == 0 && B_INSTR % 2 == 0, "load groups come in pairs");
  const int r_in = lane / NCH, pc = lane % NCH;
  const int voff[2] = {r_in * Kb + ((pc ^ ((r_in / RPB) % NCH)) << 4),
                       r_in * Kb + ((pc ^ ((4 + r_in / RPB) % NCH)) << 4)};
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  // Every operand of a load but the lane offset is wave-uniform and computed
  // from readfirstlane'd values, so it stays in SGPRs.
  const unsigned lds_ring = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(
      static_cast<int>(reinterpret_cast<uintptr_t>(static_cast<unsigned char*>(ring)))));
  const unsigned lds_bias = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(
      static_cast<int>(reinterpret_cast<uintptr_t>(&sbias[0][0]))));
  const int Kb_u = __builtin_amdgcn_readfirstlane(Kb);
  // load q of slice ks (A rows first, then W rows) of the tile with
  // descriptors (ra, rb) into ring stage su
  auto issue_one = [&](i32x4_t ra, i32x4_t rb, int su, int ks, int q) {
    const int kb = ks * ROWB;
    if (q < A_INSTR) {
      const int grp = wave_u * A_INSTR + q;
      dma16(ra, lds_ring + su * A_BYTES + grp * 1024, voff[q & 1], kb + grp * RPI * Kb_u);
    } else {
      const int grp = wave_u * B_INSTR + (q - A_INSTR);
      dma16(rb, lds_ring + B_RING + su * B_BYTES + grp * 1024, voff[(q - A_INSTR) & 1],
            kb + grp * RPI * Kb_u);
    }
  };
  // the tile's bias (256 floats, zeros past N) into bias slot bs; one wave
  // loads it, the others see it after the barrier that follows its wait
  auto issue_bias = [&](i32x4_t rbias, int bs) {
    if (wave_u == 0) dma16(rbias, lds_bias + bs * 1024, lane * 16, 0);
  };

  // fragment reads: lane -> row frow of a 32-row tile, 16-byte chunk
  // 2*kk + fch.  Tile rows start at multiples of 32, so the swizzle is
  // (frow / RPB) % NCH for every tile and the offsets per k-step are shared
  // by all tiles (the tile's row offset is an immediate).
  const int frow = lane & 31, fch = lane >> 5, fsw = (frow / RPB) % NCH;
  int a_off[KSTEPS], b_off[KSTEPS];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk) {
    a_off[kk] = (wm * WM + frow) * ROWB + (((2 * kk + fch) ^ fsw) << 4);
    b_off[kk] = B_RING + (wn * WN + frow) * ROWB + (((2 * kk + fch) ^ fsw) << 4);
  }
  auto frag_a = [&](int su, int i, int kk) {
    return *reinterpret_cast<const u32x4_t*>(ring + a_off[kk] + su * A_BYTES + i * 32 * ROWB);
  };
  auto frag_b = [&](int su, int j, int kk) {
    return *reinterpret_cast<const u32x4_t*>(ring + b_off[kk] + su * B_BYTES + j * 32 * ROWB);
  };

  f32x16_t acc[TM][TN];
  // Early free (two-stage rings of four-wave workgroups): once every wave
  // has read the last fragments of slice kt (a barrier after the reads of
  // its last k-step), the stage receives slice kt+2 while that k-step
  // multiplies, so the next barrier waits only for slice kt+1 and up to two
  // slices are in flight.  The extra barrier per slice pays off where two
  // workgroups share a CU (one multiplies while the other waits); with one
  // eight-wave workgroup per CU it costs more than it gains (measured on
  // MI355X: -5 % and +10-18 % per product).  Otherwise slice kt+STAGES-1 is
  // loaded into the stage freed at the top of the iteration.
  constexpr bool EF = STAGES == 2 && NW == 4;
  constexpr int AHEAD = EF ? 2 : STAGES - 1;  // slices between the one multiplied and the one loaded
  static_assert(!EF || KSTEPS >= 2, "early free needs two k-steps per slice");
  // Fragments of k-step kk+1 are read while k-step kk multiplies.  Without
  // early free, the loads of the slice STAGES-1 ahead go out over the first
  // two k-steps: issued all in the first, they queue behind every other
  // wave's loads before the wave reaches its first MFMA (measured on MI355X:
  // two k-steps beat one, three and four by 2-5 %).
  constexpr int LOAD_STEPS = KSTEPS < 2 ? KSTEPS : 2;
  constexpr int PER_STEP = (LOADS + LOAD_STEPS - 1) / LOAD_STEPS;
  auto compute = [&](int su, i32x4_t la, i32x4_t lb, int lsu, int lks, bool do_load) {
    u32x4_t fa[2][TM], fb[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[0][i] = frag_a(su, i, 0);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[0][j] = frag_b(su, j, 0);
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < KSTEPS) {
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[cur ^ 1][i] = frag_a(su, i, kk + 1);
#pragma unroll
        for (int j = 0; j < TN; ++j) fb[cur ^ 1][j] = frag_b(su, j, kk + 1);
      }
      if constexpr (!EF) {
#pragma unroll
        for (int q = kk * PER_STEP; q < (kk + 1) * PER_STEP && q < LOADS; ++q) issue_one(la, lb, lsu, lks, q);
      }
      // keep the reads of k-step kk+1 ahead of the MFMAs of k-step kk (left
      // alone, the scheduler sinks each read next to its first use and the
      // MFMAs wait on LDS latency at every k-step)
      __builtin_amdgcn_sched_barrier(0);
      // early free: the last k-step's MFMAs go out with the loads of slice
      // kt+2 between them, so the matrix pipe starts before the loads queue
      constexpr int LP = (LOADS + TM * TN - 1) / (TM * TN);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          Mma<T>::run(acc[i][j], fb[cur][j], fa[cur][i]);  // C^T tile
          if constexpr (EF) {
            if (kk == KSTEPS - 1 && do_load) {
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int q = (i * TN + j) * LP; q < (i * TN + j + 1) * LP && q < LOADS; ++q)
                issue_one(la, lb, lsu, lks, q);
              __builtin_amdgcn_sched_barrier(0);
            }
          }
        }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (EF) {
        if (kk == KSTEPS - 2) {
          lds_barrier();  // every wave has read its last fragments of stage su
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  const EpiCtx<T, KIND> ec = make_epi<T, KIND>(e, M, N);
  // The ring streams slices without a break across this workgroup's tiles:
  // while slice kt of a tile is multiplied, slice kt+AHEAD is loaded, which
  // near the end of a tile is one of the first slices of the next.  With
  // early free, the next tile's slice 1 waits for the epilogue (its stage is
  // the staging space) and slices past the last tile are not loaded; deeper
  // rings keep the number of loads per iteration fixed with a harmless
  // reload of the current tile's slice 0.
  const int stride = PERSIST ? static_cast<int>(gridDim.x) : total;
  int t = blockIdx.x;
  if (KT < (EF ? 2 : STAGES - 1)) return;  // the launcher picks another ring for such a short K
  i32x4_t ra, rb, rbias, na, nb, nbias;
  tile_rsrc(t, ra, rb, rbias);
  issue_bias(rbias, 0);
#pragma unroll
  for (int s = 0; s < AHEAD; ++s)
#pragma unroll
    for (int q = 0; q < LOADS; ++q) issue_one(ra, rb, s, s, q);
  // stage su holds the slice being multiplied; bs the bias slot of tile t
  int su = 0, bs = 0;
  for (int it = 0; t < total; t += stride, ++it) {
    const bool has_next = PERSIST && t + stride < total;
    if (has_next) tile_rsrc(t + stride, na, nb, nbias);
    int tm, tn;
    tile_of(t, tiles_m, tiles_n, tm, tn);
    const int m_base = tm * BM, n_base = tn * BN;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    for (int kt = 0; kt < KT; ++kt) {
      // every wave's slice kt has landed once each wave has waited for its
      // own loads of it: vector-memory operations complete in issue order,
      // so it waits until only the operations issued after them remain (one
      // load group per slice, plus at most one bias load, which only makes
      // the wait stricter).  The first slices of a later tile were issued
      // before the previous tile's epilogue, whose stores then need not
      // complete before the tile starts multiplying.
      // (without early free slices 0..AHEAD-1; with it only slice 0, as
      // slice 1 goes out after the epilogue)
      const bool after_epi = PERSIST && it > 0 && kt < (EF ? 1 : AHEAD);
      if constexpr (EF) {
        if (kt + 1 < KT || has_next) {
          if (after_epi) wait_vm<cmin(LOADS + EPI_OPS, 63)>();
          else wait_vm<LOADS>();  // slice kt+1 was issued after slice kt
        } else {
          wait_vm<0>();
        }
      } else {
        if (after_epi) wait_vm<cmin(LOADS * (STAGES - 2) + EPI_OPS, 63)>();
        else wait_vm<LOADS * (STAGES - 2)>();
      }
      __builtin_amdgcn_s_barrier();
      // without early free, the stage of slice kt-1 is free (every wave
      // passed the barrier after reading it) and receives slice kt+STAGES-1;
      // with early free, slice kt+2 goes into this slice's own stage
      const int lsu = EF ? su : (su == 0 ? STAGES - 1 : su - 1);
      const int ahead = kt + AHEAD;
      if constexpr (PERSIST) {
        const bool nxt = ahead >= KT;  // that slice belongs to the next tile
        if (nxt && has_next && ahead == KT) issue_bias(nbias, bs ^ 1);
        const bool do_load = EF ? ahead < KT || (has_next && ahead == KT) : true;
        const bool use_next = nxt && has_next;
        // one call site: the accumulators never pass through a branch; the
        // descriptors are picked component by component (scalar selects)
        i32x4_t la, lb;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          la[c] = __builtin_amdgcn_readfirstlane(use_next ? na[c] : ra[c]);
          lb[c] = __builtin_amdgcn_readfirstlane(use_next ? nb[c] : rb[c]);
        }
        compute(su, la, lb, lsu, ahead < KT ? ahead : (use_next ? ahead - KT : 0), do_load);
      } else {
        compute(su, ra, rb, lsu, ahead < KT ? ahead : 0, !EF || ahead < KT);
      }
      su = su == STAGES - 1 ? 0 : su + 1;
    }
    unsigned char* reg;
    const int fs = su == 0 ? STAGES - 1 : su - 1;  // the stage of the tile's last slice
    if constexpr (PERSIST) {
      // the stage of the tile's last slice becomes this wave's staging space
      lds_barrier();
      reg = wave < REG_IN_A ? ring + fs * A_BYTES + wave * REGION
                            : ring + B_RING + fs * B_BYTES + (wave - REG_IN_A) * REGION;
    } else {
      wait_vm<0>();  // no load may still target the ring
      lds_barrier();
      reg = ring + wave * REGION;
    }
    // a pass covers EC columns (at most 64: 128-byte staged rows for bf16)
    // so that only a few accumulator tiles are live at a time
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j0 = 0; j0 < TN; j0 += EC / 32) {
#pragma unroll
        for (int r0 = 0; r0 < 32; r0 += HS) {
          epilogue_strip<T, KIND, EC, HS>(e, ec, M, N, m_base + wm * WM + 32 * i, n_base + wn * WN + 32 * j0,
                                          lane, &sbias[bs][wn * WN + 32 * j0],
                                          *reinterpret_cast<const f32x16_t(*)[EC / 32]>(&acc[i][j0]), reg, r0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    if (has_next) {
      if constexpr (EF) {
        // the staging space is free again in every wave: the next tile's
        // slice 1 goes into it
        lds_barrier();
#pragma unroll
        for (int q = 0; q < LOADS; ++q) issue_one(na, nb, fs, 1, q);
      }
      ra = na;
      rb = nb;
      bs ^= 1;
    }
  }
  wait_vm<0>();  // no load may still target this workgroup's LDS
}

// Compute units of the current device (cached per device).
static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// persist: launch only as many workgroups as fit on the device at once; each
// loops over tiles (t, t + grid, ...) with its load ring streaming on across
// tile boundaries.  Otherwise one workgroup per tile.
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int ROWB, int KIND, bool PERSIST>
static hipError_t gemm_launch_as(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                                 hipStream_t st) {
  auto kern = gemm_kernel<T, BM, BN, WAVES_M, WAVES_N, STAGES, ROWB, KIND, PERSIST>;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  int grid = tiles;
  if (PERSIST) {
    // resident workgroups per CU, limited by LDS (160 KiB per CU): the ring,
    // the two bias slots and alignment slack; register use allows more
    constexpr int kLds = STAGES * (BM + BN) * ROWB + 2 * 1024 + 1024;
    constexpr int per_cu = kLds * 2 <= 160 * 1024 ? 2 : 1;
    grid = std::min(tiles, per_cu * device_cus());
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * WAVES_M * WAVES_N), 0, st, static_cast<const T*>(A),
                     static_cast<const T*>(W), M, N, K, e);
  return hipGetLastError();
}

template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int ROWB, int KIND>
static hipError_t gemm_launch(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                              bool persist, hipStream_t st) {
  return persist ? gemm_launch_as<T, BM, BN, WAVES_M, WAVES_N, STAGES, ROWB, KIND, true>(A, W, M, N, K, e, st)
                 : gemm_launch_as<T, BM, BN, WAVES_M, WAVES_N, STAGES, ROWB, KIND, false>(A, W, M, N, K, e, st);
}

// Tile choice.  Every configuration uses the same MFMA and visits k in the
// same order, so the choice never changes a result bit.
int g_gemm_variant = -1;  // test hook: force a variant (-1 = by shape)

// Persistent 256 x 256 launches whose last round of tiles would leave CUs
// idle: the whole rounds keep the 256 x 256 tiles (rows [0, M1)), and the
// rows left over go to a second launch of 256 x 128 tiles, at most one per
// CU, so that no CU runs a last round alone (M = 40960, N = 1024: 640 tiles
// on 256 CUs would take three rounds; 512 tiles and then 256 half-size
// tiles take about 2.6).  Each output row belongs to one tile of one launch
// and every configuration sums k in the same order: the bits do not change.
// Only for epilogues whose rows map one to one onto the output rows.
template <typename T, int KIND>
static hipError_t gemm_balanced(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                                hipStream_t st) {
  constexpr bool kRowMapped = KIND == EPI_BIAS || KIND == EPI_GELU || KIND == EPI_SILU || KIND == EPI_GATE ||
                              KIND == EPI_RESIDUAL;
  const int cus = device_cus();
  const long tn = (N + 255) / 256;
  const long tiles = static_cast<long>((M + 255) / 256) * tn;
  const long rounds = tiles / cus, rem = tiles - rounds * cus;
  const long m1_tiles = rounds * cus / tn;
  const int M1 = static_cast<int>(m1_tiles * 256), M2 = M - M1;
  const long tiles2 = static_cast<long>((M2 + 255) / 256) * ((N + 127) / 128);
  const bool split = kRowMapped && !(KIND == EPI_RESIDUAL && (e.out_idx || e.resid_copy)) && rounds > 0 &&
                     rem > 0 && M1 > 0 && M2 > 0 && tiles2 <= cus;
  if (!split) return gemm_launch<T, 256, 256, 2, 4, 2, 128, KIND>(A, W, M, N, K, e, true, st);
  hipError_t err = gemm_launch<T, 256, 256, 2, 4, 2, 128, KIND>(A, W, M1, N, K, e, true, st);
  if (err != hipSuccess) return err;
  EpiArgs e2 = e;
  const size_t off = static_cast<size_t>(M1) * N;
  if constexpr (KIND == EPI_RESIDUAL || KIND == EPI_GATE) {
    e2.out = static_cast<float*>(e.out) + off;
    e2.resid = e.resid + off;
    if constexpr (KIND == EPI_GATE) e2.gate = static_cast<const T*>(e.gate) + static_cast<size_t>(M1) * e.gate_ld;
  } else {
    e2.out = static_cast<T*>(e.out) + off;
  }
  const void* A2 = static_cast<const T*>(A) + static_cast<size_t>(M1) * K;
  return gemm_launch<T, 256, 128, 2, 2, 3, 128, KIND>(A2, W, M2, N, K, e2, false, st);
}

template <typename T, int KIND>
static hipError_t gemm_pick(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                            hipStream_t st) {
  const bool by_shape = g_gemm_variant < 0;
  constexpr bool kResid = KIND == EPI_RESIDUAL || KIND == EPI_GATE;
  constexpr bool kAct = KIND == EPI_GELU || KIND == EPI_SILU;
  int v = g_gemm_variant;
  if (v < 0) {
    // measured on MI355X over the MAR-L schedule's shapes (d_model 1024, M
    // from 3200 to 40960): 128 x 128 tiles with a three-stage ring when
    // there are at most 256 of them; 128 x 128 tiles with two workgroups per
    // CU (early free) for the fp32 residual products and the bias products
    // in the middle range, where they balance better; otherwise 256 x 256
    // tiles with a two-stage ring of 128-byte slices, launched persistent
    // once there are several tiles per CU.  Products too small to give
    // even 128 tiles of 128 x 128 (the diffusion head's, a few hundred
    // rows) take 64 x 64 tiles, four times as many workgroups; at most 256
    // tiles of 128 x 128 with the fp32 residual epilogue (the cached
    // blocks' projections at 3200 rows) run eight waves per tile; very wide
    // products on few rows (the head's modulation product, N = 33280 on
    // under 2048 rows) run persistent 128 x 128 tiles, two per CU.
    const long big = static_cast<long>((M + 255) / 256) * ((N + 255) / 256);
    const long small = static_cast<long>((M + 127) / 128) * ((N + 127) / 128);
    if (small < 128)
      v = 6;
    else if (small <= 256)
      v = kResid ? 7 : 1;
    else if (N >= 8192 && M <= 2048)
      v = 12;
    else if (kResid)
      v = big <= 512 ? 4 : 8;
    else if (big <= 512)
      v = kAct || big <= 256 ? 0 : 4;
    else
      v = big <= 1280 ? 0 : 8;
  }
  // variants 8..15: the configurations of 0..7 launched persistent
  const bool persist = v >= 8;
  if (persist) v -= 8;
  // a ring needs a minimum number of slices per tile (two for the two-stage
  // rings, which load two slices ahead; S-1 for S stages): short K takes
  // 128 x 128 tiles with 64-byte slices (K * sizeof(T) is a multiple of 128)
  static const int kMinSlices[8] = {2, 2, 2, 2, 2, 3, 2, 2}, kRowB[8] = {128, 128, 128, 128, 128, 64, 128, 128};
  if (K * static_cast<int>(sizeof(T)) / kRowB[v] < kMinSlices[v]) v = 8;
  switch (v) {
    case 8: return gemm_launch<T, 128, 128, 2, 2, 2, 64, KIND>(A, W, M, N, K, e, persist, st);
    case 7: return gemm_launch<T, 128, 128, 2, 4, 3, 128, KIND>(A, W, M, N, K, e, persist, st);
    case 0:
      if (persist && by_shape) return gemm_balanced<T, KIND>(A, W, M, N, K, e, st);
      return gemm_launch<T, 256, 256, 2, 4, 2, 128, KIND>(A, W, M, N, K, e, persist, st);
    case 1: return gemm_launch<T, 128, 128, 2, 2, 3, 128, KIND>(A, W, M, N, K, e, persist, st);
    case 2: return gemm_launch<T, 256, 128, 2, 2, 3, 128, KIND>(A, W, M, N, K, e, persist, st);
    case 3: return gemm_launch<T, 128, 256, 2, 2, 3, 128, KIND>(A, W, M, N, K, e, persist, st);
    case 5: return gemm_launch<T, 256, 256, 2, 4, 4, 64, KIND>(A, W, M, N, K, e, persist, st);
    case 6: return gemm_launch<T, 64, 64, 2, 2, 3, 128, KIND>(A, W, M, N, K, e, persist, st);
    default: return gemm_launch<T, 128, 128, 2, 2, 2, 128, KIND>(A, W, M, N, K, e, persist, st);
  }
}

template <typename T>
static hipError_t gemm_kind(const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                            hipStream_t st) {
  switch (e.kind) {
    case EPI_BIAS: return gemm_pick<T, EPI_BIAS>(A, W, M, N, K, e, st);
    case EPI_GELU: return gemm_pick<T, EPI_GELU>(A, W, M, N, K, e, st);
    case EPI_RESIDUAL: return gemm_pick<T, EPI_RESIDUAL>(A, W, M, N, K, e, st);
    case EPI_QKV: return gemm_pick<T, EPI_QKV>(A, W, M, N, K, e, st);
    default: break;
  }
  // the diffusion head's epilogues exist for bf16 operands only
  if constexpr (std::is_same<T, bf16_t>::value) {
    switch (e.kind) {
      case EPI_SILU: return gemm_pick<T, EPI_SILU>(A, W, M, N, K, e, st);
      case EPI_GATE: return gemm_pick<T, EPI_GATE>(A, W, M, N, K, e, st);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

void set_gemm_variant(int v) { g_gemm_variant = v; }

hipError_t launch_gemm(int dtype, const void* A, const void* W, int M, int N, int K,
                       const EpiArgs& e_in, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  if (N % 8) return hipErrorInvalidValue;  // epilogue stores whole 16-byte chunks
  EpiArgs e = e_in;
  if (e.kind == EPI_QKV || (e.kind == EPI_RESIDUAL && e.out_idx)) {
    if (e.per_slot < 1) return hipErrorInvalidValue;
    const Divisor dv = make_divisor(static_cast<uint32_t>(e.per_slot));
    e.slot_magic = dv.magic;
    e.slot_shift = dv.shift;
  }
  if (e.kind == EPI_QKV) {
    if (e.d_head < 1 || e.d_model % 32 || e.n_offset % 32) return hipErrorInvalidValue;
    const Divisor dh = make_divisor(static_cast<uint32_t>(e.d_head));
    e.head_magic = dh.magic;
    e.head_shift = dh.shift;
  }
  // 32-bit buffer offsets: a tile's operand rows and every output must span
  // less than 2 GiB
  const size_t es = dtype == DT_BF16 ? 2 : 4;
  const size_t lim = 1ull << 31;
  if (static_cast<size_t>(256) * K * es >= lim || (K * es) % 128) return hipErrorInvalidValue;
  if (static_cast<size_t>(M) * N * 4 >= lim) return hipErrorInvalidValue;
  if (e.kind == EPI_RESIDUAL && e.out_idx &&
      static_cast<size_t>((M + e.per_slot - 1) / e.per_slot) * e.seq * N * 4 >= lim)
    return hipErrorInvalidValue;
  if (e.kind == EPI_QKV && static_cast<size_t>((M + e.per_slot - 1) / e.per_slot) * e.n_heads * e.seq *
                                   e.d_head * es >= lim)
    return hipErrorInvalidValue;
  if (e.kind == EPI_GATE && (e.gate_ld < N || e.gate_ld % 4 || static_cast<size_t>(M) * e.gate_ld * es >= lim))
    return hipErrorInvalidValue;
  if (dtype == DT_BF16) return gemm_kind<bf16_t>(A, W, M, N, K, e, st);
  return gemm_kind<float>(A, W, M, N, K, e, st);
}

}  // namespace marcache
