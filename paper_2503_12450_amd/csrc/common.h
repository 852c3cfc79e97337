// Shared device helpers and launcher declarations of the cached MAR step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>

namespace marcache {

typedef uint16_t bf16_t;  // bfloat16 bits
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16, round to nearest even (the hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = static_cast<__bf16>(f);
  return __builtin_bit_cast(bf16_t, b);
}

// Element traits: storage type <-> fp32.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ float to_f(float v) { return v; }
  static __device__ __forceinline__ float from_f(float v) { return v; }
  static constexpr int kPer16B = 4;
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float to_f(bf16_t v) { return bf2f(v); }
  static __device__ __forceinline__ bf16_t from_f(float v) { return f2bf(v); }
  static constexpr int kPer16B = 8;
};

// Unpack one 16-byte vector of storage elements to fp32.
__device__ __forceinline__ void unpack16(const u32x4_t& v, float* out, const float*) {
  out[0] = __uint_as_float(v[0]);
  out[1] = __uint_as_float(v[1]);
  out[2] = __uint_as_float(v[2]);
  out[3] = __uint_as_float(v[3]);
}
__device__ __forceinline__ void unpack16(const u32x4_t& v, float* out, const bf16_t*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(v[i] << 16);
    out[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
  }
}

// Two fp32 -> two bf16 (round to nearest even) in one packed conversion.
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// Exact division by a divisor d >= 2 fixed for the launch (Granlund &
// Montgomery, "Division by invariant integers using multiplication", 1994):
// with s = 31 + ceil(log2 d) >= 32 and magic = ceil(2^s / d) < 2^32,
// floor(m / d) = (m * magic) >> s for every 0 <= m < 2^31.  d = 1 is
// encoded as magic 0 (the identity).
struct Divisor {
  uint32_t magic;
  int shift;  // s - 32
};
inline Divisor make_divisor(uint32_t d) {
  if (d <= 1) return Divisor{0u, 0};
  int l = 0;
  while ((1ull << l) < d) ++l;
  const int s = 31 + l;
  const uint64_t magic = ((1ull << s) + d - 1) / d;
  return Divisor{static_cast<uint32_t>(magic), s - 32};
}
__device__ __forceinline__ int div_by(int m, uint32_t magic, int shift) {
  return magic ? static_cast<int>(__umulhi(static_cast<uint32_t>(m), magic) >> shift) : m;
}

// Sum across the 64 lanes of a wave; every lane gets the total.  Within each
// row of 16 lanes, four DPP steps (lane swaps 1 and 2 in a quad, then the
// half-row and row mirrors) leave the row's sum in every lane without a trip
// through LDS; the four row sums are then added in row order.  The order of
// additions is fixed, so the result is deterministic.
template <int CTRL>
__device__ __forceinline__ float dpp_shift_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_shift_add<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v = dpp_shift_add<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v = dpp_shift_add<0x141>(v);  // row_half_mirror
  v = dpp_shift_add<0x140>(v);  // row_mirror
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return ((r0 + r1) + r2) + r3;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// The thread-local message behind mar_last_error(): cleared at the start of
// every C entry point, set by a failing one (never allocates).
void abi_clear_error();
int abi_fail_v(int status, const char* fmt, va_list ap);

// ---------------------------------------------------------------------------
// Launchers (host side).  All return hipSuccess or the launch error.
// Rows of a "slot-mapped" matrix: row m belongs to slot m / per_slot and to
// token idx[m] (or m % per_slot when idx is null) of that slot.
// ---------------------------------------------------------------------------

// Row LayerNorm: out[m] = LN(src_row(m)) in dtype, optional fp32 copy of the
// source row.  src_row(m) = src[(m / per_slot) * seq + tok(m)] where tok(m)
// = idx[m] when idx is given, else m % per_slot (then seq must equal
// per_slot).  src is fp32 when src_f32, else the storage dtype.
hipError_t launch_layernorm(int dtype, const void* src, bool src_f32, const int32_t* idx,
                            int per_slot, int seq, int M, int D, const float* w,
                            const float* b, float eps, float* copy_f32, void* out,
                            hipStream_t st);

// Epilogue kinds of the matrix product C = A W^T (A [M,K], W [N,K]).
enum EpiKind {
  EPI_BIAS = 0,      // out[m, n] = C + bias[n]                        (dtype)
  EPI_GELU = 1,      // out[m, n] = gelu(C + bias[n])                  (dtype)
  EPI_RESIDUAL = 2,  // out[row(m), n] = resid[m, n] + C + bias[n]     (fp32)
  EPI_QKV = 3,       // split into q rows and key/value cache rows     (dtype)
  EPI_SILU = 4,      // out[m, n] = silu(C + bias[n])                  (bf16 only)
  EPI_GATE = 5       // out[m, n] = resid[m, n] + gate[m, n] (C + bias[n])  (fp32; bf16 only)
};

struct EpiArgs {
  int kind;
  const float* bias;
  void* out;           // BIAS/GELU: [M, N]; RESIDUAL: fp32 rows; QKV: q [M, D]
  const float* resid;  // RESIDUAL: fp32 [M, N] (may equal out when no remap)
  // RESIDUAL remap: when out_idx is non-null, row m goes to
  //   out[(m / per_slot) * seq + out_idx[m]] (the output-cache scatter);
  //   resid_copy (nullable) also receives the row at m.
  const int32_t* out_idx;
  float* resid_copy;
  // QKV: n_global = n + n_offset selects q (< D), k (< 2D) or v; keys go to
  // k_cache[slot][head][tok][d], values to v_cache[slot][head][tok][d] (and
  // v_copy, same layout), with slot/tok from the row mapping (idx or dense).
  int n_offset;
  int d_model, n_heads, d_head, seq, per_slot;
  // m / per_slot = umulhi(m, slot_magic) >> slot_shift (set by launch_gemm)
  uint32_t slot_magic;
  int slot_shift;
  // QKV: r / d_head = umulhi(r, head_magic) >> head_shift (set by launch_gemm)
  uint32_t head_magic;
  int head_shift;
  const int32_t* idx;
  void* k_cache;
  void* v_cache;
  void* v_copy;  // nullable: value rows again, [slot][head][tok][d]
  // GATE: gate[m, n] = gate[m * gate_ld + n] in the storage dtype
  const void* gate;
  int gate_ld;
};

hipError_t launch_gemm(int dtype, const void* A, const void* W, int M, int N, int K,
                       const EpiArgs& epi, hipStream_t st);
void set_gemm_variant(int v);  // -1: by shape

// Attention of per_slot queries per slot against the seq keys of the slot:
// q, out [n_slots * per_slot, D] (head h at columns h*dh..); k and v
// [n_slots, H, seq, dh].
hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v, void* out,
                            int n_slots, int H, int seq, int dh, int per_slot,
                            hipStream_t st);

// Cosine scores of value rows (Eq. 8) for [n_slots, H, seq, dh] layouts;
// optionally copies v_cur into v_ref afterwards.
hipError_t launch_scores(int dtype, const void* v_cur, void* v_ref, int n_slots, int H,
                         int seq, int dh, double* scores, bool update_ref, hipStream_t st);

// The n least similar tokens of each slot (the n most similar when
// `largest`), ascending.
hipError_t launch_select(const double* scores, int n_slots, int seq, int n, bool largest, int32_t* idx,
                         hipStream_t st);

// Guidance with the condition cache over `count` fp32 elements.
hipError_t launch_cfg(int op, const float* c, const float* u, float* stored, float scale,
                      float* guided, float* u_out, size_t count, hipStream_t st);

}  // namespace marcache
