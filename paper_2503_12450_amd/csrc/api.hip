// C ABI of the cached MAR step: workspace layout, argument/state checks and
// the kernel sequence of one step (full, token-cached, or given rows).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <new>
#include <vector>

#include "../../include/mar_cache.h"
#include "../../include/mar_kernels.h"
#include "common.h"

using namespace marcache;

// The last error of this thread, in a fixed buffer: reporting an error never
// allocates, so nothing can throw across the C boundary from here.
static thread_local char g_err[512];

namespace marcache {
void abi_clear_error() { g_err[0] = '\0'; }
int abi_fail_v(int s, const char* fmt, va_list ap) {
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  return s;
}
}  // namespace marcache

namespace {

void clear_error() { abi_clear_error(); }

mar_status fail(mar_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  abi_fail_v(s, fmt, ap);
  va_end(ap);
  return s;
}

mar_status hip_fail(hipError_t e, const char* what) {
  return fail(MAR_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define MAR_HIP(call, what)                          \
  do {                                               \
    hipError_t e_ = (call);                          \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int kMaxSeq = 4096;
constexpr int kMaxModel = 2048;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
size_t elem_size(int dtype) { return dtype == MAR_BF16 ? 2 : 4; }

mar_status check_dims(const mar_dims* d) {
  if (!d) return fail(MAR_E_ARG, "dims is NULL");
  if (d->dtype != MAR_F32 && d->dtype != MAR_BF16) return fail(MAR_E_ARG, "unknown dtype %d", d->dtype);
  if (d->n_layers < 1) return fail(MAR_E_SHAPE, "n_layers must be >= 1");
  if (d->n_heads < 1 || d->d_model < 1 || d->d_model % d->n_heads)
    return fail(MAR_E_SHAPE, "d_model must be a positive multiple of n_heads");
  const int dh = d->d_model / d->n_heads;
  if (dh % 16 || dh > 128) return fail(MAR_E_SHAPE, "d_head %d must be a multiple of 16, <= 128", dh);
  if (d->d_model % 64 || d->d_model > kMaxModel)
    return fail(MAR_E_SHAPE, "d_model %d must be a multiple of 64, <= %d", d->d_model, kMaxModel);
  if (d->d_mlp < 64 || d->d_mlp % 64) return fail(MAR_E_SHAPE, "d_mlp must be a positive multiple of 64");
  if (d->seq_len < 1 || d->seq_len > kMaxSeq) return fail(MAR_E_SHAPE, "seq_len must be in [1, %d]", kMaxSeq);
  if (d->max_slots < 1) return fail(MAR_E_SHAPE, "max_slots must be >= 1");
  if (d->full_prefix < 0 || d->full_prefix >= d->n_layers)
    return fail(MAR_E_SHAPE, "full_prefix must be in [0, n_layers)");
  if (!(d->ln_eps > 0.f)) return fail(MAR_E_ARG, "ln_eps must be positive");
  if (d->score_source != MAR_SCORE_VALUES && d->score_source != MAR_SCORE_FEATURES)
    return fail(MAR_E_ARG, "unknown score_source %d", d->score_source);
  if (d->fresh_kv != 0 && d->fresh_kv != 1) return fail(MAR_E_ARG, "fresh_kv must be 0 or 1");
  // The products address operands and outputs through buffer descriptors
  // with 32-bit byte offsets (launch_gemm refuses anything that reaches
  // 2 GiB).  Checked here, so that every step mar_workspace_bytes accepts
  // runs to the end once its arguments pass: the widest product of a full
  // step writes max_slots * seq_len rows of max(3 d_model, d_mlp) columns
  // (fp32-sized in the check); the key/value caches, the output cache and
  // the residual stream are narrower; a weight panel is 256 rows of K.
  const size_t es = d->dtype == MAR_BF16 ? 2 : 4;
  const size_t lim = size_t(1) << 31;
  const size_t rows = static_cast<size_t>(d->max_slots) * d->seq_len;
  const size_t widest = std::max<size_t>(3 * static_cast<size_t>(d->d_model), d->d_mlp);
  if (rows * widest * 4 >= lim)
    return fail(MAR_E_SHAPE,
                "max_slots * seq_len * max(3 d_model, d_mlp) * 4 = %zu bytes reaches 2 GiB (32-bit offsets); "
                "use fewer slots per cache",
                rows * widest * 4);
  if (size_t(256) * std::max(d->d_model, d->d_mlp) * es >= lim)
    return fail(MAR_E_SHAPE, "d_mlp %d too large for 32-bit weight offsets", d->d_mlp);
  return MAR_OK;
}

struct LayerPtrs {
  void *qkv_w, *proj_w, *fc1_w, *fc2_w;
  float *ln1_w, *ln1_b, *ln2_w, *ln2_b, *qkv_b, *proj_b, *fc1_b, *fc2_b;
  void *kc, *vc;  // key/value caches [max_slots, H, S, dh] (blocks >= P)
};

struct Layout {
  size_t total = 0;
  std::vector<size_t> w_off;  // per layer base of its parameters
  size_t w_qkv = 0, w_proj = 0, w_fc1 = 0, w_fc2 = 0, b_ln1w = 0, b_ln1b = 0, b_ln2w = 0, b_ln2b = 0,
         b_qkv = 0, b_proj = 0, b_fc1 = 0, b_fc2 = 0, layer_bytes = 0;
  std::vector<size_t> kc_off, vc_off;
  size_t vref = 0, fref = 0, Y = 0, cres = 0;
  size_t h = 0, c = 0, a = 0, q = 0, o = 0, f = 0, ktmp = 0, vtmp = 0, vcur = 0, scores = 0, idx = 0;
};

Layout make_layout(const mar_dims& d) {
  Layout L;
  const size_t es = elem_size(d.dtype);
  const size_t D = d.d_model, F = d.d_mlp, S = d.seq_len, NS = d.max_slots;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  // parameter block (offsets relative to the layer base)
  L.w_qkv = take(3 * D * D * es);
  L.w_proj = take(D * D * es);
  L.w_fc1 = take(F * D * es);
  L.w_fc2 = take(D * F * es);
  L.b_ln1w = take(D * 4);
  L.b_ln1b = take(D * 4);
  L.b_ln2w = take(D * 4);
  L.b_ln2b = take(D * 4);
  L.b_qkv = take(3 * D * 4);
  L.b_proj = take(D * 4);
  L.b_fc1 = take(F * 4);
  L.b_fc2 = take(D * 4);
  L.layer_bytes = o;
  o = 0;
  for (int l = 0; l < d.n_layers; ++l) L.w_off.push_back(take(L.layer_bytes));
  const size_t rows = NS * S;
  L.kc_off.assign(d.n_layers, 0);
  L.vc_off.assign(d.n_layers, 0);
  for (int l = d.full_prefix; l < d.n_layers; ++l) {
    L.kc_off[l] = take(rows * D * es);
    L.vc_off[l] = take(rows * D * es);
  }
  L.vref = take(rows * D * es);
  // feature reference: block P-1's fp32 output rows, or x when P = 0
  if (d.score_source == MAR_SCORE_FEATURES) L.fref = take(rows * D * (d.full_prefix == 0 ? es : 4));
  L.Y = take(rows * D * 4);
  const size_t pairs = (NS + 1) / 2;
  L.cres = take(pairs * S * D * 4);
  L.h = take(rows * D * 4);
  L.c = take(rows * D * 4);
  L.a = take(rows * D * es);
  L.q = take(rows * D * es);
  L.o = take(rows * D * es);
  L.f = take(rows * F * es);
  L.ktmp = take(rows * D * es);
  L.vtmp = take(rows * D * es);
  L.vcur = take(rows * D * es);
  L.scores = take(rows * 8);
  L.idx = take(rows * 4);
  L.total = o;
  return L;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

struct mar_cache {
  mar_dims d;
  Layout lay;
  unsigned char* ws;
  std::vector<LayerPtrs> layers;
  std::vector<unsigned char> filled;  // per slot
  std::vector<unsigned char> stored;  // per guidance pair
  int pairs;
  // profiler: event pairs around every launch of one kernel class
  int prof_kind = -1;
  std::vector<hipEvent_t> events;  // pool, reused across sessions
  size_t ev_used = 0;
  double prof_flops = 0.0, prof_bytes = 0.0;
  int64_t prof_launches = 0;

  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(ws + off); }

  ~mar_cache() {
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
  }
};

namespace {

struct StepCtx {
  mar_cache* h;
  hipStream_t st;
  int n;          // slots in this call
  int slot0;
  size_t es;
  int D, H, dh, F, S, L, P, dtype;
  float eps;
  long slot_elems;  // H * S * dh
};

#define STEP_HIP(call, what)                         \
  do {                                               \
    hipError_t e_ = (call);                          \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// Runs `launch`; when the handle profiles `kind`, brackets it with a pair of
// events on the stream and adds the launch's algorithmic work.
// A session times at most this many launches (an event pair each); later
// launches of the class run untimed, so a long session cannot exhaust events.
constexpr size_t kMaxTimedLaunches = size_t(1) << 18;

template <class F>
mar_status timed(mar_cache* h, hipStream_t st, int kind, double flops, double bytes, F&& launch,
                 const char* what) {
  const bool on = h->prof_kind == kind && h->ev_used / 2 < kMaxTimedLaunches;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (on) {
    while (h->events.size() < h->ev_used + 2) {
      hipEvent_t e;
      hipError_t err = hipEventCreate(&e);
      if (err != hipSuccess) return hip_fail(err, "profiler event");
      try {
        h->events.push_back(e);
      } catch (const std::bad_alloc&) {
        (void)hipEventDestroy(e);
        return fail(MAR_E_HOST, "out of host memory");
      }
    }
    e0 = h->events[h->ev_used];
    e1 = h->events[h->ev_used + 1];
    hipError_t err = hipEventRecord(e0, st);
    if (err != hipSuccess) return hip_fail(err, "profiler event");
  }
  hipError_t err = launch();
  if (err != hipSuccess) return hip_fail(err, what);
  if (on) {
    err = hipEventRecord(e1, st);
    if (err != hipSuccess) return hip_fail(err, "profiler event");
    h->ev_used += 2;
    h->prof_flops += flops;
    h->prof_bytes += bytes;
    h->prof_launches += 1;
  }
  return MAR_OK;
}

#define TIMED(kind, flops, bytes, call, what)                                                      \
  do {                                                                                             \
    mar_status s_ = timed(c.h, c.st, (kind), static_cast<double>(flops), static_cast<double>(bytes), \
                          [&]() { return (call); }, (what));                                      \
    if (s_ != MAR_OK) return s_;                                                                   \
  } while (0)

double gemm_bytes(double M, double N, double K, double es, double out_es, bool resid) {
  return (M * K + N * K) * es + M * N * out_es + (resid ? M * N * 4.0 : 0.0);
}

template <typename P> P* offset(void* base, long elems, size_t es) {
  return reinterpret_cast<P*>(static_cast<unsigned char*>(base) + elems * es);
}

// One block on every row of the call's slots.  The block input is x
// (storage dtype) for block 0, else the fp32 residual stream h.
mar_status dense_block(const StepCtx& c, int l, bool from_x, const void* x, void* kdst, void* vdst,
                       void* vcopy, float* final_out) {
  const mar_cache* hd = c.h;
  const LayerPtrs& w = hd->layers[l];
  const int M = c.n * c.S;
  const double Md = M, D = c.D, F = c.F, es = static_cast<double>(c.es);
  float* h = hd->at<float>(hd->lay.h);
  void* a = hd->at<void>(hd->lay.a);
  void* q = hd->at<void>(hd->lay.q);
  void* o = hd->at<void>(hd->lay.o);
  void* f = hd->at<void>(hd->lay.f);
  TIMED(MAR_PROF_LAYERNORM, 0, Md * D * ((from_x ? es : 4.0) + es + (from_x ? 4.0 : 0.0)),
        launch_layernorm(c.dtype, from_x ? x : static_cast<const void*>(h), !from_x, nullptr, c.S, c.S, M,
                         c.D, w.ln1_w, w.ln1_b, c.eps, from_x ? h : nullptr, a, c.st),
        "layernorm");
  EpiArgs e{};
  e.kind = EPI_QKV;
  e.bias = w.qkv_b;
  e.out = q;
  e.n_offset = 0;
  e.d_model = c.D;
  e.n_heads = c.H;
  e.d_head = c.dh;
  e.seq = c.S;
  e.per_slot = c.S;
  e.idx = nullptr;
  e.k_cache = kdst;
  e.v_cache = vdst;
  e.v_copy = vcopy;
  TIMED(MAR_PROF_QKV, 2.0 * Md * 3 * D * D, gemm_bytes(Md, 3 * D, D, es, es, false),
        launch_gemm(c.dtype, a, w.qkv_w, M, 3 * c.D, c.D, e, c.st), "qkv gemm");
  TIMED(MAR_PROF_ATTENTION, 4.0 * Md * c.S * D, 4.0 * Md * D * es,
        launch_attention(c.dtype, q, kdst, vdst, o, c.n, c.H, c.S, c.dh, c.S, c.st), "attention");
  EpiArgs r{};
  r.kind = EPI_RESIDUAL;
  r.bias = w.proj_b;
  r.out = h;
  r.resid = h;
  TIMED(MAR_PROF_PROJ, 2.0 * Md * D * D, gemm_bytes(Md, D, D, es, 4.0, true),
        launch_gemm(c.dtype, o, w.proj_w, M, c.D, c.D, r, c.st), "proj gemm");
  TIMED(MAR_PROF_LAYERNORM, 0, Md * D * (4.0 + es),
        launch_layernorm(c.dtype, h, true, nullptr, c.S, c.S, M, c.D, w.ln2_w, w.ln2_b, c.eps, nullptr, a,
                         c.st),
        "layernorm");
  EpiArgs g{};
  g.kind = EPI_GELU;
  g.bias = w.fc1_b;
  g.out = f;
  TIMED(MAR_PROF_FC1, 2.0 * Md * F * D, gemm_bytes(Md, F, D, es, es, false),
        launch_gemm(c.dtype, a, w.fc1_w, M, c.F, c.D, g, c.st), "fc1 gemm");
  EpiArgs r2{};
  r2.kind = EPI_RESIDUAL;
  r2.bias = w.fc2_b;
  r2.out = final_out ? final_out : h;
  r2.resid = h;
  TIMED(MAR_PROF_FC2, 2.0 * Md * D * F, gemm_bytes(Md, D, F, es, 4.0, true),
        launch_gemm(c.dtype, f, w.fc2_w, M, c.D, c.F, r2, c.st), "fc2 gemm");
  return MAR_OK;
}

// One cached block (Eq. 9) on the compact rows of the selected tokens.
// The fp32 residual rows are in c, LN1 of them already in a.
mar_status cached_block(const StepCtx& c, int l, int N, const int32_t* idx, float* Yslot) {
  const mar_cache* hd = c.h;
  const LayerPtrs& w = hd->layers[l];
  const int M = c.n * N;
  const double Md = M, D = c.D, F = c.F, es = static_cast<double>(c.es);
  float* cres = hd->at<float>(hd->lay.c);
  void* a = hd->at<void>(hd->lay.a);
  void* q = hd->at<void>(hd->lay.q);
  void* o = hd->at<void>(hd->lay.o);
  void* f = hd->at<void>(hd->lay.f);
  void* kc = offset<void>(w.kc, static_cast<long>(c.slot0) * c.slot_elems, c.es);
  void* vc = offset<void>(w.vc, static_cast<long>(c.slot0) * c.slot_elems, c.es);
  EpiArgs e{};
  e.kind = EPI_QKV;
  e.bias = w.qkv_b;
  e.out = q;
  e.d_model = c.D;
  e.n_heads = c.H;
  e.d_head = c.dh;
  e.seq = c.S;
  e.per_slot = N;
  e.idx = idx;
  e.k_cache = kc;
  e.v_cache = vc;
  TIMED(MAR_PROF_QKV, 2.0 * Md * 3 * D * D, gemm_bytes(Md, 3 * D, D, es, es, false),
        launch_gemm(c.dtype, a, w.qkv_w, M, 3 * c.D, c.D, e, c.st), "qkv gemm (selected rows)");
  // kernel boundary: every scattered key/value row lands before attention
  TIMED(MAR_PROF_ATTENTION, 4.0 * Md * c.S * D, 2.0 * Md * D * es + 2.0 * c.n * c.S * D * es,
        launch_attention(c.dtype, q, kc, vc, o, c.n, c.H, c.S, c.dh, N, c.st), "partial attention");
  EpiArgs r{};
  r.kind = EPI_RESIDUAL;
  r.bias = w.proj_b;
  r.out = cres;
  r.resid = cres;
  TIMED(MAR_PROF_PROJ, 2.0 * Md * D * D, gemm_bytes(Md, D, D, es, 4.0, true),
        launch_gemm(c.dtype, o, w.proj_w, M, c.D, c.D, r, c.st), "proj gemm (selected rows)");
  TIMED(MAR_PROF_LAYERNORM, 0, Md * D * (4.0 + es),
        launch_layernorm(c.dtype, cres, true, nullptr, M, M, M, c.D, w.ln2_w, w.ln2_b, c.eps, nullptr, a,
                         c.st),
        "layernorm");
  EpiArgs g{};
  g.kind = EPI_GELU;
  g.bias = w.fc1_b;
  g.out = f;
  TIMED(MAR_PROF_FC1, 2.0 * Md * F * D, gemm_bytes(Md, F, D, es, es, false),
        launch_gemm(c.dtype, a, w.fc1_w, M, c.F, c.D, g, c.st), "fc1 gemm (selected rows)");
  EpiArgs r2{};
  r2.kind = EPI_RESIDUAL;
  r2.bias = w.fc2_b;
  r2.resid = cres;
  if (l == c.L - 1) {  // scatter the fresh rows into the output cache
    r2.out = Yslot;
    r2.out_idx = idx;
    r2.per_slot = N;
    r2.seq = c.S;
    r2.resid_copy = nullptr;
  } else {
    r2.out = cres;
  }
  TIMED(MAR_PROF_FC2, 2.0 * Md * D * F, gemm_bytes(Md, D, F, es, 4.0, true),
        launch_gemm(c.dtype, f, w.fc2_w, M, c.D, c.F, r2, c.st), "fc2 gemm (selected rows)");
  if (l < c.L - 1) {
    const LayerPtrs& wn = hd->layers[l + 1];
    TIMED(MAR_PROF_LAYERNORM, 0, Md * D * (4.0 + es),
          launch_layernorm(c.dtype, cres, true, nullptr, M, M, M, c.D, wn.ln1_w, wn.ln1_b, c.eps, nullptr,
                           a, c.st),
          "layernorm");
  }
  return MAR_OK;
}

}  // namespace

extern "C" {

const char* mar_last_error(void) { return g_err; }

size_t mar_workspace_bytes(const mar_dims* dims) {
  if (check_dims(dims) != MAR_OK) return 0;
  try {
    return make_layout(*dims).total;
  } catch (const std::bad_alloc&) {
    fail(MAR_E_HOST, "out of host memory");
    return 0;
  }
}

namespace {

mar_status cache_init(const mar_dims* dims, const mar_block_weights* blocks, void* workspace,
                      size_t workspace_bytes, void* stream, mar_cache** out) {
  if (!out) return fail(MAR_E_ARG, "out is NULL");
  *out = nullptr;
  mar_status s = check_dims(dims);
  if (s != MAR_OK) return s;
  if (!blocks) return fail(MAR_E_ARG, "blocks is NULL");
  if (!workspace) return fail(MAR_E_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(MAR_E_WORKSPACE, "workspace must be %zu-byte aligned", kAlign);
  Layout lay = make_layout(*dims);
  if (workspace_bytes < lay.total)
    return fail(MAR_E_WORKSPACE, "workspace holds %zu bytes, %zu needed", workspace_bytes, lay.total);
  for (int l = 0; l < dims->n_layers; ++l) {
    const mar_block_weights& b = blocks[l];
    const void* ptrs[] = {b.ln1_w, b.ln1_b, b.qkv_w, b.qkv_b, b.proj_w, b.proj_b,
                          b.ln2_w, b.ln2_b, b.fc1_w, b.fc1_b, b.fc2_w, b.fc2_b};
    for (const void* p : ptrs)
      if (!p) return fail(MAR_E_ARG, "block %d has a NULL parameter pointer", l);
  }
  std::unique_ptr<mar_cache> h(new (std::nothrow) mar_cache);
  if (!h) return fail(MAR_E_HOST, "out of host memory");
  h->d = *dims;
  h->lay = lay;
  h->ws = static_cast<unsigned char*>(workspace);
  h->filled.assign(dims->max_slots, 0);
  h->pairs = (dims->max_slots + 1) / 2;
  h->stored.assign(h->pairs, 0);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t es = elem_size(dims->dtype);
  const size_t D = dims->d_model, F = dims->d_mlp;
  for (int l = 0; l < dims->n_layers; ++l) {
    const size_t base = lay.w_off[l];
    LayerPtrs p{};
    p.qkv_w = h->at<void>(base + lay.w_qkv);
    p.proj_w = h->at<void>(base + lay.w_proj);
    p.fc1_w = h->at<void>(base + lay.w_fc1);
    p.fc2_w = h->at<void>(base + lay.w_fc2);
    p.ln1_w = h->at<float>(base + lay.b_ln1w);
    p.ln1_b = h->at<float>(base + lay.b_ln1b);
    p.ln2_w = h->at<float>(base + lay.b_ln2w);
    p.ln2_b = h->at<float>(base + lay.b_ln2b);
    p.qkv_b = h->at<float>(base + lay.b_qkv);
    p.proj_b = h->at<float>(base + lay.b_proj);
    p.fc1_b = h->at<float>(base + lay.b_fc1);
    p.fc2_b = h->at<float>(base + lay.b_fc2);
    p.kc = l >= dims->full_prefix ? h->at<void>(lay.kc_off[l]) : nullptr;
    p.vc = l >= dims->full_prefix ? h->at<void>(lay.vc_off[l]) : nullptr;
    h->layers.push_back(p);
    const mar_block_weights& b = blocks[l];
    struct Cp { void* dst; const void* src; size_t bytes; } cps[] = {
        {p.qkv_w, b.qkv_w, 3 * D * D * es}, {p.proj_w, b.proj_w, D * D * es},
        {p.fc1_w, b.fc1_w, F * D * es},     {p.fc2_w, b.fc2_w, D * F * es},
        {p.ln1_w, b.ln1_w, D * 4},          {p.ln1_b, b.ln1_b, D * 4},
        {p.ln2_w, b.ln2_w, D * 4},          {p.ln2_b, b.ln2_b, D * 4},
        {p.qkv_b, b.qkv_b, 3 * D * 4},      {p.proj_b, b.proj_b, D * 4},
        {p.fc1_b, b.fc1_b, F * 4},          {p.fc2_b, b.fc2_b, D * 4}};
    for (const Cp& cp : cps) {
      hipError_t e = hipMemcpyAsync(cp.dst, cp.src, cp.bytes, hipMemcpyDeviceToDevice, st);
      if (e != hipSuccess) return hip_fail(e, "weight copy");
    }
  }
  *out = h.release();
  return MAR_OK;
}

}  // namespace

mar_status mar_cache_init(const mar_dims* dims, const mar_block_weights* blocks, void* workspace,
                          size_t workspace_bytes, void* stream, mar_cache** out) {
  clear_error();
  try {
    return cache_init(dims, blocks, workspace, workspace_bytes, stream, out);
  } catch (const std::bad_alloc&) {
    return fail(MAR_E_HOST, "out of host memory");
  }
}

mar_status mar_cache_destroy(mar_cache* cache) {
  delete cache;
  return MAR_OK;
}

const float* mar_output(const mar_cache* cache) {
  if (!cache) return nullptr;
  return cache->at<float>(cache->lay.Y);
}

mar_status mar_step(mar_cache* cache, const void* x, float* y, int32_t slot0, int32_t n_slots,
                    int32_t mode, int32_t n_recompute, int32_t* sel_idx, void* stream) {
  clear_error();
  if (!cache) return fail(MAR_E_ARG, "cache is NULL");
  const mar_dims& d = cache->d;
  if (!x) return fail(MAR_E_ARG, "x is NULL");
  if (!aligned16(x)) return fail(MAR_E_ARG, "x must be 16-byte aligned");
  if (slot0 < 0 || n_slots < 1 || slot0 > d.max_slots - n_slots)
    return fail(MAR_E_ARG, "slots [%d, %d) outside [0, %d)", slot0, slot0 + n_slots, d.max_slots);
  if (mode != MAR_FULL && mode != MAR_TOKEN_CACHED && mode != MAR_TOKEN_GIVEN &&
      mode != MAR_TOKEN_CACHED_MOST_SIMILAR)
    return fail(MAR_E_ARG, "unknown mode %d", mode);
  const int S = d.seq_len;
  const int N = n_recompute;
  if (mode != MAR_FULL) {
    if (N < 0 || N > S) return fail(MAR_E_ARG, "n_recompute %d outside [0, %d]", N, S);
    for (int b = slot0; b < slot0 + n_slots; ++b)
      if (!cache->filled[b]) return fail(MAR_E_STATE, "slot %d has no cache yet: run MAR_FULL first", b);
    if (mode == MAR_TOKEN_GIVEN) {
      if (N > 0 && !sel_idx) return fail(MAR_E_ARG, "MAR_TOKEN_GIVEN needs the host index array");
      for (int b = 0; b < n_slots; ++b)
        for (int i = 0; i < N; ++i) {
          const int32_t t = sel_idx[static_cast<long>(b) * N + i];
          if (t < 0 || t >= S) return fail(MAR_E_ARG, "index %d of slot %d outside [0, %d)", t, b, S);
          if (i > 0 && t <= sel_idx[static_cast<long>(b) * N + i - 1])
            return fail(MAR_E_ARG, "indices of slot %d must be strictly ascending", b);
        }
    }
  }
  {
    hipError_t e = hipPeekAtLastError();
    if (e != hipSuccess) return hip_fail(e, "earlier device error");
  }
  StepCtx c;
  c.h = cache;
  c.st = static_cast<hipStream_t>(stream);
  c.n = n_slots;
  c.slot0 = slot0;
  c.es = elem_size(d.dtype);
  c.D = d.d_model;
  c.H = d.n_heads;
  c.dh = d.d_model / d.n_heads;
  c.F = d.d_mlp;
  c.S = S;
  c.L = d.n_layers;
  c.P = d.full_prefix;
  c.dtype = d.dtype;
  c.eps = d.ln_eps;
  c.slot_elems = static_cast<long>(c.H) * S * c.dh;
  const Layout& lay = cache->lay;
  const long slot_off = static_cast<long>(slot0) * c.slot_elems;
  void* vref = offset<void>(cache->at<void>(lay.vref), slot_off, c.es);
  float* Yslot = cache->at<float>(lay.Y) + static_cast<long>(slot0) * S * c.D;
  void* ktmp = cache->at<void>(lay.ktmp);
  void* vtmp = cache->at<void>(lay.vtmp);
  void* vcur = cache->at<void>(lay.vcur);
  const int score_layer = c.P > 0 ? c.P - 1 : 0;
  // feature scoring (Sec. 4.4 alternative): block P-1's fp32 output rows,
  // or x (storage dtype) when P = 0, against the previous step's
  const bool features = d.score_source == MAR_SCORE_FEATURES;
  const size_t fes = c.P == 0 ? c.es : 4;
  void* fref = features ? static_cast<char*>(cache->at<void>(lay.fref)) +
                              static_cast<size_t>(slot0) * S * c.D * fes
                        : nullptr;
  float* hbuf = cache->at<float>(lay.h);
  const size_t feat_bytes = static_cast<size_t>(n_slots) * S * c.D * fes;
  mar_status s;

  if (mode == MAR_FULL) {
    if (features && c.P == 0)
      STEP_HIP(hipMemcpyAsync(fref, x, feat_bytes, hipMemcpyDeviceToDevice, c.st), "feature reference");
    for (int l = 0; l < c.L; ++l) {
      // keys and values [slot, head, token, d]: into the cache from block P
      // on; the scoring block's values go to the scoring reference (as a
      // second copy when that block is cached too)
      void* kd = l >= c.P ? offset<void>(cache->layers[l].kc, slot_off, c.es) : ktmp;
      void* vd = l >= c.P ? offset<void>(cache->layers[l].vc, slot_off, c.es)
                          : (l == score_layer ? vref : vtmp);
      void* vcopy = l == score_layer && l >= c.P ? vref : nullptr;
      s = dense_block(c, l, l == 0, x, kd, vd, vcopy, l == c.L - 1 ? Yslot : nullptr);
      if (s != MAR_OK) return s;
      if (features && l == c.P - 1)
        STEP_HIP(hipMemcpyAsync(fref, hbuf, feat_bytes, hipMemcpyDeviceToDevice, c.st), "feature reference");
    }
    for (int b = slot0; b < slot0 + n_slots; ++b) cache->filled[b] = 1;
  } else {
    const int Mfull = n_slots * S;
    if (c.P == 0 && !features) {
      // score pass: value rows of block 0 from x
      const LayerPtrs& w = cache->layers[0];
      void* a = cache->at<void>(lay.a);
      TIMED(MAR_PROF_LAYERNORM, 0, 2.0 * Mfull * c.D * c.es,
            launch_layernorm(c.dtype, x, false, nullptr, S, S, Mfull, c.D, w.ln1_w, w.ln1_b, c.eps, nullptr,
                             a, c.st),
            "layernorm");
      EpiArgs e{};
      e.kind = EPI_QKV;
      e.bias = w.qkv_b + 2 * c.D;
      e.out = nullptr;
      e.n_offset = 2 * c.D;
      e.d_model = c.D;
      e.n_heads = c.H;
      e.d_head = c.dh;
      e.seq = S;
      e.per_slot = S;
      e.v_cache = vcur;  // value rows only, for scoring
      e.v_copy = nullptr;
      const void* wv = offset<const void>(w.qkv_w, 2L * c.D * c.D, c.es);
      TIMED(MAR_PROF_QKV, 2.0 * Mfull * c.D * c.D,
            gemm_bytes(Mfull, c.D, c.D, static_cast<double>(c.es), static_cast<double>(c.es), false),
            launch_gemm(c.dtype, a, wv, Mfull, c.D, c.D, e, c.st), "value gemm");
    } else {
      for (int l = 0; l < c.P; ++l) {
        s = dense_block(c, l, l == 0, x, ktmp, l == score_layer ? vcur : vtmp, nullptr, nullptr);
        if (s != MAR_OK) return s;
      }
    }
    double* scores = cache->at<double>(lay.scores);
    int32_t* idx = cache->at<int32_t>(lay.idx);
    if (features) {
      // a feature row is one "head" of width D in the scoring layout
      TIMED(MAR_PROF_SCORES, 0, 3.0 * Mfull * c.D * static_cast<double>(fes) + 8.0 * Mfull,
            launch_scores(c.P == 0 ? c.dtype : static_cast<int>(DT_F32), c.P == 0 ? x : hbuf, fref, n_slots,
                          1, S, c.D, scores, true, c.st),
            "feature scores");
    } else {
      TIMED(MAR_PROF_SCORES, 0, 3.0 * Mfull * c.D * c.es + 8.0 * Mfull,
            launch_scores(c.dtype, vcur, vref, n_slots, c.H, S, c.dh, scores, true, c.st), "scores");
    }
    if (mode == MAR_TOKEN_CACHED || mode == MAR_TOKEN_CACHED_MOST_SIMILAR) {
      TIMED(MAR_PROF_SELECT, 0, 8.0 * Mfull + 4.0 * n_slots * N,
            launch_select(scores, n_slots, S, N, mode == MAR_TOKEN_CACHED_MOST_SIMILAR, idx, c.st), "select");
      if (sel_idx && N > 0)
        STEP_HIP(hipMemcpyAsync(sel_idx, idx, sizeof(int32_t) * n_slots * N, hipMemcpyDeviceToDevice,
                                c.st),
                 "index copy");
    } else if (N > 0) {
      STEP_HIP(hipMemcpyAsync(idx, sel_idx, sizeof(int32_t) * n_slots * N, hipMemcpyHostToDevice, c.st),
               "index upload");
    }
    if (d.fresh_kv) {
      // keys/values of every row at block P from this step's block P-1
      // output (x when P = 0), before the computed rows replace their own
      const LayerPtrs& w = cache->layers[c.P];
      const bool from_x = c.P == 0;
      void* a = cache->at<void>(lay.a);
      TIMED(MAR_PROF_LAYERNORM, 0, static_cast<double>(Mfull) * c.D * ((from_x ? c.es : 4.0) + c.es),
            launch_layernorm(c.dtype, from_x ? x : static_cast<const void*>(hbuf), !from_x, nullptr, S, S, Mfull,
                             c.D, w.ln1_w, w.ln1_b, c.eps, nullptr, a, c.st),
            "layernorm (fresh keys/values)");
      EpiArgs e{};
      e.kind = EPI_QKV;
      e.bias = w.qkv_b + c.D;
      e.out = nullptr;
      e.n_offset = c.D;
      e.d_model = c.D;
      e.n_heads = c.H;
      e.d_head = c.dh;
      e.seq = S;
      e.per_slot = S;
      e.k_cache = offset<void>(w.kc, slot_off, c.es);
      e.v_cache = offset<void>(w.vc, slot_off, c.es);
      const void* wkv = offset<const void>(w.qkv_w, static_cast<long>(c.D) * c.D, c.es);
      TIMED(MAR_PROF_QKV, 2.0 * Mfull * 2 * c.D * c.D,
            gemm_bytes(Mfull, 2 * c.D, c.D, static_cast<double>(c.es), static_cast<double>(c.es), false),
            launch_gemm(c.dtype, a, wkv, Mfull, 2 * c.D, c.D, e, c.st), "key/value gemm (fresh)");
    }
    if (N > 0) {
      const int Msel = n_slots * N;
      const LayerPtrs& w = cache->layers[c.P];
      const bool from_x = c.P == 0;
      TIMED(MAR_PROF_LAYERNORM, 0, static_cast<double>(Msel) * c.D * ((from_x ? c.es : 4.0) + 4.0 + c.es),
            launch_layernorm(c.dtype, from_x ? x : cache->at<void>(lay.h), !from_x, idx, N, S, Msel, c.D,
                             w.ln1_w, w.ln1_b, c.eps, cache->at<float>(lay.c), cache->at<void>(lay.a), c.st),
            "gather layernorm");
      for (int l = c.P; l < c.L; ++l) {
        s = cached_block(c, l, N, idx, Yslot);
        if (s != MAR_OK) return s;
      }
    }
  }
  if (y)
    STEP_HIP(hipMemcpyAsync(y, Yslot, sizeof(float) * n_slots * S * c.D, hipMemcpyDeviceToDevice, c.st),
             "output copy");
  return MAR_OK;
}

mar_status mar_cfg_combine(mar_cache* cache, const float* y_cond, const float* y_uncond, int32_t pair0,
                           int32_t n_pairs, int32_t op, float scale, float* guided, float* uncond_out,
                           void* stream) {
  clear_error();
  if (!cache) return fail(MAR_E_ARG, "cache is NULL");
  if (op != MAR_CFG_STORE && op != MAR_CFG_REUSE) return fail(MAR_E_ARG, "unknown op %d", op);
  if (!y_cond || !guided) return fail(MAR_E_ARG, "y_cond and guided are required");
  if (op == MAR_CFG_STORE && !y_uncond) return fail(MAR_E_ARG, "STORE needs y_uncond");
  if (pair0 < 0 || n_pairs < 1 || pair0 > cache->pairs - n_pairs)
    return fail(MAR_E_ARG, "pairs [%d, %d) outside [0, %d)", pair0, pair0 + n_pairs, cache->pairs);
  const float* ptrs[] = {y_cond, op == MAR_CFG_STORE ? y_uncond : y_cond, guided,
                         uncond_out ? uncond_out : guided};
  for (const float* p : ptrs)
    if (!aligned16(p)) return fail(MAR_E_ARG, "guidance buffers must be 16-byte aligned");
  if (op == MAR_CFG_REUSE)
    for (int p = pair0; p < pair0 + n_pairs; ++p)
      if (!cache->stored[p]) return fail(MAR_E_STATE, "pair %d has no stored residual: STORE first", p);
  {
    hipError_t e = hipPeekAtLastError();
    if (e != hipSuccess) return hip_fail(e, "earlier device error");
  }
  const size_t per = static_cast<size_t>(cache->d.seq_len) * cache->d.d_model;
  float* stored = cache->at<float>(cache->lay.cres) + static_cast<size_t>(pair0) * per;
  const double count = static_cast<double>(per) * n_pairs;
  const double bytes = count * 4.0 * (op == MAR_CFG_STORE ? 4 : 3) + (uncond_out ? count * 4.0 : 0.0);
  hipStream_t st = static_cast<hipStream_t>(stream);
  mar_status ts = timed(cache, st, MAR_PROF_CFG, 0.0, bytes,
                        [&]() {
                          return launch_cfg(op, y_cond, y_uncond, stored, scale, guided, uncond_out,
                                            per * n_pairs, st);
                        },
                        "guidance");
  if (ts != MAR_OK) return ts;
  if (op == MAR_CFG_STORE)
    for (int p = pair0; p < pair0 + n_pairs; ++p) cache->stored[p] = 1;
  return MAR_OK;
}

mar_status mar_profile_start(mar_cache* cache, int32_t kind) {
  clear_error();
  if (!cache) return fail(MAR_E_ARG, "cache is NULL");
  if (kind < 0 || kind >= MAR_PROF_KINDS) return fail(MAR_E_ARG, "unknown kernel class %d", kind);
  cache->prof_kind = kind;
  cache->ev_used = 0;
  cache->prof_flops = cache->prof_bytes = 0.0;
  cache->prof_launches = 0;
  return MAR_OK;
}

mar_status mar_profile_stop(mar_cache* cache, double* ms_total, int64_t* launches, double* flops,
                            double* bytes) {
  clear_error();
  if (!cache) return fail(MAR_E_ARG, "cache is NULL");
  if (cache->prof_kind < 0) return fail(MAR_E_STATE, "no profile session");
  double total = 0.0;
  if (cache->ev_used > 0) {
    MAR_HIP(hipEventSynchronize(cache->events[cache->ev_used - 1]), "profiler event");
    for (size_t i = 0; i < cache->ev_used; i += 2) {
      float ms = 0.f;
      MAR_HIP(hipEventElapsedTime(&ms, cache->events[i], cache->events[i + 1]), "profiler event");
      total += ms;
    }
  }
  if (ms_total) *ms_total = total;
  if (launches) *launches = cache->prof_launches;
  if (flops) *flops = cache->prof_flops;
  if (bytes) *bytes = cache->prof_bytes;
  cache->prof_kind = -1;
  cache->ev_used = 0;
  return MAR_OK;
}

// ---------------------------------------------------------------------------
// Per-kernel entry points
// ---------------------------------------------------------------------------

static mar_status check_dtype(int32_t dtype) {
  if (dtype != MAR_F32 && dtype != MAR_BF16) return fail(MAR_E_ARG, "unknown dtype %d", dtype);
  return MAR_OK;
}

mar_status mar_k_layernorm(int32_t dtype, const void* src, int32_t src_f32, const int32_t* idx,
                           int32_t per_slot, int32_t seq, int32_t m, int32_t d, const float* w,
                           const float* b, float eps, float* copy_f32, void* out, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!src || !w || !b || !out) return fail(MAR_E_ARG, "NULL pointer");
  if (m < 0 || d < 8 || d % 8 || d > kMaxModel) return fail(MAR_E_SHAPE, "d must be a multiple of 8, <= %d", kMaxModel);
  if (per_slot < 1 || seq < 1 || (!idx && per_slot != seq)) return fail(MAR_E_SHAPE, "bad row mapping");
  if (!aligned16(src) || !aligned16(out) || !aligned16(w) || !aligned16(b) || (copy_f32 && !aligned16(copy_f32)))
    return fail(MAR_E_ARG, "buffers must be 16-byte aligned");
  MAR_HIP(launch_layernorm(dtype, src, src_f32 != 0, idx, per_slot, seq, m, d, w, b, eps, copy_f32, out,
                           static_cast<hipStream_t>(stream)),
          "layernorm");
  return MAR_OK;
}

mar_status mar_k_linear(int32_t dtype, int32_t act, const void* a, const void* w, const float* bias,
                        int32_t m, int32_t n, int32_t k, void* out, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!a || !w || !bias || !out) return fail(MAR_E_ARG, "NULL pointer");
  if (m < 0 || k < 64 || k % 64) return fail(MAR_E_SHAPE, "k must be a positive multiple of 64");
  if (n < 8 || n % 8) return fail(MAR_E_SHAPE, "n must be a positive multiple of 8");
  if (!aligned16(a) || !aligned16(w) || !aligned16(out)) return fail(MAR_E_ARG, "operands must be 16-byte aligned");
  EpiArgs e{};
  e.kind = act ? EPI_GELU : EPI_BIAS;
  e.bias = bias;
  e.out = out;
  MAR_HIP(launch_gemm(dtype, a, w, m, n, k, e, static_cast<hipStream_t>(stream)), "gemm");
  return MAR_OK;
}

mar_status mar_k_linear_residual(int32_t dtype, const void* a, const void* w, const float* bias, int32_t m,
                                 int32_t n, int32_t k, const float* resid, float* out,
                                 const int32_t* out_idx, int32_t per_slot, int32_t seq,
                                 float* resid_copy, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!a || !w || !bias || !resid || !out) return fail(MAR_E_ARG, "NULL pointer");
  if (m < 0 || k < 64 || k % 64) return fail(MAR_E_SHAPE, "k must be a positive multiple of 64");
  if (n < 8 || n % 8) return fail(MAR_E_SHAPE, "n must be a positive multiple of 8");
  if (out_idx && (per_slot < 1 || seq < 1)) return fail(MAR_E_SHAPE, "bad row mapping");
  if (!aligned16(a) || !aligned16(w) || !aligned16(resid) || !aligned16(out) ||
      (resid_copy && !aligned16(resid_copy)))
    return fail(MAR_E_ARG, "operands must be 16-byte aligned");
  EpiArgs e{};
  e.kind = EPI_RESIDUAL;
  e.bias = bias;
  e.out = out;
  e.resid = resid;
  e.out_idx = out_idx;
  e.per_slot = per_slot;
  e.seq = seq;
  e.resid_copy = resid_copy;
  MAR_HIP(launch_gemm(dtype, a, w, m, n, k, e, static_cast<hipStream_t>(stream)), "gemm");
  return MAR_OK;
}

mar_status mar_k_qkv(int32_t dtype, const void* a, const void* w, const float* bias, int32_t m,
                     int32_t n_cols, int32_t n_offset, int32_t d_model, int32_t n_heads, int32_t seq,
                     int32_t per_slot, const int32_t* idx, void* q_out, void* k_cache, void* v_cache,
                     void* v_copy, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!a || !w || !bias) return fail(MAR_E_ARG, "NULL pointer");
  if (n_heads < 1 || d_model % 64 || d_model % n_heads || (d_model / n_heads) % 16)
    return fail(MAR_E_SHAPE, "bad d_model/n_heads");
  if (n_offset < 0 || n_offset % 32 || n_cols < 8 || n_cols % 8 || n_offset + n_cols > 3 * d_model)
    return fail(MAR_E_SHAPE, "bad columns");
  if (per_slot < 1 || seq < 1 || (!idx && per_slot != seq)) return fail(MAR_E_SHAPE, "bad row mapping");
  const bool has_q = n_offset < d_model, has_k = n_offset < 2 * d_model && n_offset + n_cols > d_model,
             has_v = n_offset + n_cols > 2 * d_model;
  if ((has_q && !q_out) || (has_k && !k_cache) || (has_v && !v_cache && !v_copy))
    return fail(MAR_E_ARG, "missing output for the requested columns");
  if (!aligned16(a) || !aligned16(w) || !aligned16(q_out) || !aligned16(k_cache) || !aligned16(v_cache) ||
      !aligned16(v_copy))
    return fail(MAR_E_ARG, "operands must be 16-byte aligned");
  EpiArgs e{};
  e.kind = EPI_QKV;
  e.bias = bias;
  e.out = q_out;
  e.n_offset = n_offset;
  e.d_model = d_model;
  e.n_heads = n_heads;
  e.d_head = d_model / n_heads;
  e.seq = seq;
  e.per_slot = per_slot;
  e.idx = idx;
  e.k_cache = k_cache;
  e.v_cache = v_cache;
  e.v_copy = v_copy;
  MAR_HIP(launch_gemm(dtype, a, w, m, n_cols, d_model, e, static_cast<hipStream_t>(stream)), "gemm");
  return MAR_OK;
}

mar_status mar_k_attention(int32_t dtype, const void* q, const void* k, const void* v, void* out,
                           int32_t n_slots, int32_t n_heads, int32_t seq, int32_t d_head,
                           int32_t per_slot, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!q || !k || !v || !out) return fail(MAR_E_ARG, "NULL pointer");
  if (n_slots < 0 || n_heads < 1 || seq < 1 || per_slot < 0) return fail(MAR_E_SHAPE, "bad sizes");
  if (d_head % 16 || d_head < 16 || d_head > 128) return fail(MAR_E_SHAPE, "d_head must be 16..128, multiple of 16");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(MAR_E_ARG, "buffers must be 16-byte aligned");
  MAR_HIP(launch_attention(dtype, q, k, v, out, n_slots, n_heads, seq, d_head, per_slot,
                           static_cast<hipStream_t>(stream)),
          "attention");
  return MAR_OK;
}

mar_status mar_k_scores(int32_t dtype, const void* v_cur, void* v_ref, int32_t n_slots, int32_t n_heads,
                        int32_t seq, int32_t d_head, double* scores, int32_t update_ref, void* stream) {
  clear_error();
  if (check_dtype(dtype) != MAR_OK) return MAR_E_ARG;
  if (!v_cur || !v_ref || !scores) return fail(MAR_E_ARG, "NULL pointer");
  if (n_slots < 0 || n_heads < 1 || seq < 1 || d_head < 8 || d_head % 8)
    return fail(MAR_E_SHAPE, "bad sizes");
  if (!aligned16(v_cur) || !aligned16(v_ref)) return fail(MAR_E_ARG, "buffers must be 16-byte aligned");
  MAR_HIP(launch_scores(dtype, v_cur, v_ref, n_slots, n_heads, seq, d_head, scores, update_ref != 0,
                        static_cast<hipStream_t>(stream)),
          "scores");
  return MAR_OK;
}

static mar_status select_rule(const double* scores, int32_t n_slots, int32_t seq, int32_t n, bool largest,
                              int32_t* idx, void* stream) {
  clear_error();
  if (!scores || (!idx && n > 0 && n_slots > 0)) return fail(MAR_E_ARG, "NULL pointer");
  if (n_slots < 0 || seq < 1 || seq > kMaxSeq || n < 0 || n > seq) return fail(MAR_E_SHAPE, "bad sizes");
  MAR_HIP(launch_select(scores, n_slots, seq, n, largest, idx, static_cast<hipStream_t>(stream)), "select");
  return MAR_OK;
}

mar_status mar_k_select(const double* scores, int32_t n_slots, int32_t seq, int32_t n, int32_t* idx,
                        void* stream) {
  return select_rule(scores, n_slots, seq, n, false, idx, stream);
}

mar_status mar_k_select_most_similar(const double* scores, int32_t n_slots, int32_t seq, int32_t n,
                                     int32_t* idx, void* stream) {
  return select_rule(scores, n_slots, seq, n, true, idx, stream);
}

mar_status mar_k_gemm_variant(int32_t variant) {
  clear_error();
  if (variant < -1 || variant >= MAR_GEMM_VARIANTS) return fail(MAR_E_ARG, "unknown variant %d", variant);
  set_gemm_variant(variant);
  return MAR_OK;
}

}  // extern "C"
