// C ABI entry points for the sparsified MLP, the sparsified attention and the whole
// decoder layer, plus status strings and the per-device CU count cache.
//
// Every entry point validates all arguments on the host before touching the device,
// carves its scratch buffers out of the caller's workspace and enqueues its kernels
// on the caller's stream.
#include <atomic>
#include <mutex>
#include <set>
#include <utility>
#include <string.h>
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

// Device properties, read once per device (up to 64 devices) and kept in atomics:
// concurrent first calls may both query, and store the same value.
namespace {
std::atomic<int> g_cus[64], g_lds[64];

int current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  return dev;
}

int cached_attr(std::atomic<int>* cache, hipDeviceAttribute_t attr, int fallback) {
  const int dev = current_device();
  if (dev < 64) {
    const int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, attr, dev) != hipSuccess || v <= 0) v = fallback;
  if (dev < 64) cache[dev].store(v, std::memory_order_relaxed);
  return v;
}
}  // namespace

int device_cu_count() { return cached_attr(g_cus, hipDeviceAttributeMultiprocessorCount, 256); }

int device_lds_per_block() { return cached_attr(g_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, 65536); }

hipError_t ensure_dyn_lds(const void* kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  static std::mutex mu;
  static std::set<std::pair<const void*, int>> done;
  const int dev = current_device();
  {
    std::lock_guard<std::mutex> g(mu);
    if (done.count({kern, dev})) return hipSuccess;
  }
  hipFuncAttributes fa{};
  hipError_t e = hipFuncGetAttributes(&fa, kern);
  if (e != hipSuccess) return e;
  const int limit = device_lds_per_block() - (int)fa.sharedSizeBytes;
  if ((long)bytes > (long)limit) return hipErrorInvalidValue;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, limit);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> g(mu);
  done.insert({kern, dev});
  return hipSuccess;
}

namespace {
struct Trace {
  void** events = nullptr;
  int n_pairs = 0;
  int32_t* n_launched = nullptr;
  const char* only = nullptr;   // time only launches with this label (NULL: all)
  int count = 0;                // launches of the current call
  int timed = 0;                // event pairs used by the current call
  bool open = false;            // the current launch records events
  bool started = false;         // its start event went to a kernel
  const char* labels[64] = {};
};
thread_local Trace g_trace;
}  // namespace

void trace_reset() {
  g_trace.count = 0;
  g_trace.timed = 0;
}

void trace_begin(const char* label, hipStream_t st) {
  Trace& t = g_trace;
  if (t.count < 64) t.labels[t.count] = label;
  t.open = t.events != nullptr && t.timed < t.n_pairs && (t.only == nullptr || strcmp(t.only, label) == 0);
  t.started = false;
  (void)st;
}

void trace_take(hipEvent_t* start, hipEvent_t* stop) {
  Trace& t = g_trace;
  if (!t.open) return;
  if (!t.started) *start = static_cast<hipEvent_t>(t.events[2 * t.timed]);
  *stop = static_cast<hipEvent_t>(t.events[2 * t.timed + 1]);
  t.started = true;
}

void trace_end(hipStream_t st) {
  Trace& t = g_trace;
  if (t.open) {
    if (!t.started) {   // no kernel ran: an empty interval, so both events are set
      (void)hipEventRecord(static_cast<hipEvent_t>(t.events[2 * t.timed]), st);
      (void)hipEventRecord(static_cast<hipEvent_t>(t.events[2 * t.timed + 1]), st);
    }
    ++t.timed;
    t.open = false;
  }
  ++t.count;
  if (t.n_launched) *t.n_launched = t.count;
}

}  // namespace dv

using namespace dv;

extern "C" dv_status dv_set_launch_events(void** events, int32_t n_pairs, int32_t* n_launched, const char* only) {
  if (n_pairs < 0) return DV_ERR_SHAPE;
  g_trace.events = events;
  g_trace.n_pairs = events ? n_pairs : 0;
  g_trace.n_launched = events ? n_launched : nullptr;
  g_trace.only = events ? only : nullptr;
  return DV_OK;
}

extern "C" const char* dv_launch_label(int32_t i) {
  return (i >= 0 && i < g_trace.count && i < 64) ? g_trace.labels[i] : "";
}

// ------------------------------------------------------------------ helpers
bool dv::dtype_ok(int t) { return t == DV_F16 || t == DV_F32; }
int dv::chunk_elems(int t) { return 16 / elem_bytes(t); }
bool dv::ws_ok(void* ws) { return ws != nullptr && (reinterpret_cast<uintptr_t>(ws) & 255u) == 0; }

dv_status dv::check_mlp(const dv_mlp* m) {
  if (m == nullptr || m->W1T == nullptr || m->W2T == nullptr) return DV_ERR_NULL;
  if (!dtype_ok(m->wtype)) return DV_ERR_DTYPE;
  if (m->act != DV_ACT_RELU && m->act != DV_ACT_GELU) return DV_ERR_ARG;
  if (m->d <= 0 || m->n <= 0) return DV_ERR_SHAPE;
  if (m->d % chunk_elems(m->wtype) != 0) return DV_ERR_ALIGN;
  if (!aligned16(m->W1T) || !aligned16(m->W2T)) return DV_ERR_ALIGN;
  if (m->d > kMaxWidth) return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

dv_status dv::check_attn(const dv_attn* a) {
  if (a == nullptr || a->Wq == nullptr || a->Wk == nullptr || a->Wv == nullptr || a->WoT == nullptr)
    return DV_ERR_NULL;
  if (!dtype_ok(a->wtype)) return DV_ERR_DTYPE;
  if (a->d <= 0 || a->H <= 0 || a->dh <= 0) return DV_ERR_SHAPE;
  if (a->d % chunk_elems(a->wtype) != 0) return DV_ERR_ALIGN;
  if (!aligned16(a->Wq) || !aligned16(a->Wk) || !aligned16(a->Wv) || !aligned16(a->WoT)) return DV_ERR_ALIGN;
  if (a->d > kMaxWidth || a->dh > 256) return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

dv_status dv::check_kv(const dv_kv* kv, const dv_attn* a, int B) {
  if (kv == nullptr || kv->K == nullptr || kv->V == nullptr || kv->pos == nullptr) return DV_ERR_NULL;
  if (!dtype_ok(kv->ktype)) return DV_ERR_DTYPE;
  if (kv->reserved != 0) return DV_ERR_ARG;
  if (kv->B != B || kv->H != a->H || kv->dh != a->dh || kv->cap <= 0) return DV_ERR_SHAPE;
  if ((kv->dh * elem_bytes(kv->ktype)) % 16 != 0) return DV_ERR_ALIGN;
  if (!aligned16(kv->K) || !aligned16(kv->V)) return DV_ERR_ALIGN;
  for (int b = 0; b < B; ++b)
    if (kv->pos[b] < 0 || kv->pos[b] >= kv->cap) return DV_ERR_SHAPE;
  return DV_OK;
}

dv_status dv::check_ln(const dv_ln* ln) {
  if (ln == nullptr) return DV_OK;
  const float* p[4] = {ln->g1, ln->be1, ln->g2, ln->be2};
  for (const float* q : p)
    if (q != nullptr && !aligned16(q)) return DV_ERR_ALIGN;
  if ((ln->be1 && !ln->g1) || (ln->be2 && !ln->g2)) return DV_ERR_ARG;
  if (!(ln->eps >= 0.f)) return DV_ERR_ARG;
  return DV_OK;
}

dv_status dv::validate_sets_sync(const int32_t* set, int B, int n, int range, int32_t* flag, hipStream_t st) {
  DV_LAUNCH("validate", st, launch_validate_sets(set, B, n, range, flag, st));
  int32_t bad = 0;
  if (hipMemcpyAsync(&bad, flag, sizeof(bad), hipMemcpyDeviceToHost, st) != hipSuccess) return DV_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return DV_ERR_HIP;
  return bad ? DV_ERR_INDEX : DV_OK;
}
static dv_status validate_sets(const int32_t* set, int B, int n, int range, int32_t* flag, hipStream_t st) {
  return validate_sets_sync(set, B, n, range, flag, st);
}

// The batched path: 2..kMaxBatch sequences, fp16 weights.
static constexpr int kMaxUnionN = 131072;   // the union builder marks n bytes in LDS
static bool batch_ok(int B, int wtype) { return B <= kMaxBatch && wtype == DV_F16; }

static dv_status enqueue_axpy(const char* label, int wtype, const AxpyArgs& ax, hipStream_t hs) {
  DV_LAUNCH(label, hs, launch_axpy(wtype, ax, hs));
  return DV_OK;
}

// ---------------------------------------------------------------- sparse MLP
struct MlpWs {
  float* h; float* axp; uint32_t* axc; int32_t* flag;
};

// Row-split partial sums of a gathered row-axpy of width d.
size_t dv::axpy_partial_bytes(int d) { return (size_t)kAxpyMaxRowSplit * d * sizeof(float); }

static size_t mlp_ws_layout(const dv_mlp* m, int B, int n_idx, Workspace& w, MlpWs* o) {
  o->h = w.take<float>((size_t)B * n_idx * sizeof(float));
  o->axp = w.take<float>(axpy_partial_bytes(m->d));
  o->axc = w.take<uint32_t>(kAxpyMaxSpans * sizeof(uint32_t));
  o->flag = w.take<int32_t>(sizeof(int32_t));
  return w.off;
}

extern "C" size_t dv_sparse_mlp_workspace_bytes(const dv_mlp* m, int32_t B, int32_t n_idx, int32_t idx_per_seq) {
  if (m == nullptr || m->d <= 0 || m->n <= 0 || B <= 0 || n_idx < 0 || !dtype_ok(m->wtype)) return 0;
  if (B > 1) return batch_mlp_ws(m, B, n_idx, idx_per_seq);
  Workspace w(nullptr);
  MlpWs o;
  return mlp_ws_layout(m, B, n_idx, w, &o);
}

extern "C" dv_status dv_sparse_mlp(const dv_mlp* m, const float* x, int32_t B, const int32_t* idx,
                                   int32_t n_idx, int32_t idx_per_seq, int32_t batch_mode, float* out,
                                   void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_mlp(m);
  if (st != DV_OK) return st;
  if (x == nullptr || out == nullptr || (idx == nullptr && n_idx > 0)) return DV_ERR_NULL;
  if (B <= 0 || n_idx < 0 || n_idx > m->n) return DV_ERR_SHAPE;
  if (!aligned16(x) || !aligned16(out)) return DV_ERR_ALIGN;
  if (idx_per_seq != 0 && idx_per_seq != 1) return DV_ERR_ARG;
  if (batch_mode != DV_MLP_UNION && batch_mode != DV_MLP_MASKED) return DV_ERR_ARG;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (m->b1 != nullptr && !aligned16(m->b1)) return DV_ERR_ALIGN;
  if (m->b2 != nullptr && !aligned16(m->b2)) return DV_ERR_ALIGN;
  if (B > 1 && (!batch_ok(B, m->wtype) || m->n > kMaxUnionN)) return DV_ERR_UNSUPPORTED;
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (B > 1) return batch_mlp(m, x, B, idx, n_idx, idx_per_seq, batch_mode, out, ws, ws_bytes, flags, hs);
  Workspace w(ws);
  MlpWs o;
  if (mlp_ws_layout(m, B, n_idx, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  if (flags & DV_VALIDATE) {
    st = validate_sets(idx, 1, n_idx, m->n, o.flag, hs);
    if (st != DV_OK) return st;
  }
  Fc1Args f{};
  f.d = m->d; f.k = n_idx; f.n = m->n; f.x = x; f.g = nullptr; f.be = nullptr; f.eps = 0.f;
  f.W1T = m->W1T; f.b1 = m->b1; f.set = idx; f.h = o.h; f.clear = o.axc; f.clear_n = kAxpyMaxSpans;
  f.act = m->act;
  DV_LAUNCH("fc1", hs, launch_fc1(m->wtype, f, hs));
  AxpyArgs ax{};
  ax.d = m->d; ax.nrows = n_idx; ax.M = m->W2T; ax.m_rows = m->n; ax.set = idx; ax.dh = 0;
  ax.coef = o.h; ax.resid = nullptr; ax.bias = m->b2; ax.out = out; ax.out2 = nullptr; ax.partial = o.axp;
  ax.cnt = o.axc;
  if ((st = enqueue_axpy("fc2", m->wtype, ax, hs)) != DV_OK) return st;
  return DV_OK;
}

// ---------------------------------------------------------- sparse attention
struct AttnWs {
  int32_t* heads; float* q; float* part; float* axp; uint32_t* axc; int32_t* flag;
};

static size_t attn_ws_layout(const dv_attn* a, int B, int n_heads, Workspace& w, AttnWs* o) {
  o->heads = w.take<int32_t>((size_t)B * n_heads * sizeof(int32_t));
  o->q = w.take<float>((size_t)B * n_heads * a->dh * sizeof(float));
  o->part = w.take<float>((size_t)B * n_heads * kAttnMaxSplit * (a->dh + 2) * sizeof(float));
  o->axp = w.take<float>(axpy_partial_bytes(a->d));
  o->axc = w.take<uint32_t>(kAxpyMaxSpans * sizeof(uint32_t));
  o->flag = w.take<int32_t>(sizeof(int32_t));
  return w.off;
}

extern "C" size_t dv_sparse_attn_workspace_bytes(const dv_attn* a, const dv_kv* kv, int32_t B, int32_t n_heads) {
  if (a == nullptr || kv == nullptr || a->d <= 0 || a->dh <= 0 || a->H <= 0 || B <= 0 || n_heads < 0 ||
      kv->cap <= 0 || !dtype_ok(a->wtype))
    return 0;
  if (B > 1) return batch_attn_ws(a, B, n_heads);
  Workspace w(nullptr);
  AttnWs o;
  return attn_ws_layout(a, B, n_heads, w, &o);
}

static dv_status enqueue_attention(const dv_attn* a, const dv_kv* kv, const AttnWs& o, int n_heads,
                                   float scale, hipStream_t hs, uint8_t* valid = nullptr) {
  const int pos = kv->pos[0];
  AttnArgs at{};
  at.H = a->H; at.dh = a->dh; at.cap = kv->cap; at.posb[0] = pos; at.n_heads = n_heads;
  at.chunk = attn_chunk(n_heads, pos + 1, a->dh, kv->ktype);
  at.n_split = (pos + 1 + at.chunk - 1) / at.chunk;
  at.q = o.q; at.heads = o.heads; at.K = kv->K; at.V = kv->V; at.scale = scale; at.part = o.part;
  at.valid = valid;
  DV_LAUNCH("attn", hs, launch_attn(kv->ktype, at, 1, hs));
  return DV_OK;
}

static int attn_nsplit(const dv_attn* a, const dv_kv* kv, int n_heads) {
  const int pos = kv->pos[0];
  const int ch = attn_chunk(n_heads, pos + 1, a->dh, kv->ktype);
  return (pos + 1 + ch - 1) / ch;
}

extern "C" dv_status dv_sparse_attn(const dv_attn* a, const float* x, int32_t B, const dv_kv* kv,
                                    const int32_t* heads, int32_t n_heads, float scale, float* out,
                                    void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_attn(a);
  if (st != DV_OK) return st;
  if (x == nullptr || out == nullptr || (heads == nullptr && n_heads > 0)) return DV_ERR_NULL;
  if (B <= 0 || n_heads < 0 || n_heads > a->H) return DV_ERR_SHAPE;
  st = check_kv(kv, a, B);
  if (st != DV_OK) return st;
  if (!aligned16(x) || !aligned16(out)) return DV_ERR_ALIGN;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (!isfinite(scale)) return DV_ERR_ARG;
  if (a->bo != nullptr && !aligned16(a->bo)) return DV_ERR_ALIGN;
  if (B > 1 && (!batch_ok(B, a->wtype) || a->H > kMaxUnionN)) return DV_ERR_UNSUPPORTED;
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (B > 1) return batch_attn(a, x, B, kv, heads, n_heads, scale, out, ws, ws_bytes, flags, hs);
  Workspace w(ws);
  AttnWs o;
  if (attn_ws_layout(a, B, n_heads, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  if (flags & DV_VALIDATE) {
    st = validate_sets(heads, 1, n_heads, a->H, o.flag, hs);
    if (st != DV_OK) return st;
  }
  if (n_heads == 0) {
    // MHA over the empty set is bo (or zero): one axpy over no rows writes it.
    AxpyArgs ax{};
    ax.d = a->d; ax.nrows = 0; ax.M = a->WoT; ax.m_rows = a->H * a->dh; ax.set = o.heads; ax.dh = 0;
    ax.coef = o.q; ax.bias = a->bo; ax.out = out;
    DV_LAUNCH("oproj", hs, launch_axpy(a->wtype, ax, hs));
    return DV_OK;
  }
  QkvArgs q{};
  q.d = a->d; q.H = a->H; q.dh = a->dh; q.cap = kv->cap; q.pos = kv->pos[0]; q.n_heads = n_heads;
  q.x = x;
  q.Wq = a->Wq; q.Wk = a->Wk; q.Wv = a->Wv; q.bq = a->bq; q.bk = a->bk; q.bv = a->bv;
  q.K = kv->K; q.V = kv->V; q.q = o.q; q.heads_in = heads; q.heads_ws = o.heads;
  q.clear = o.axc; q.clear_n = kAxpyMaxSpans;
  DV_LAUNCH("qkv", hs, launch_qkv(a->wtype, kv->ktype, q, hs));
  st = enqueue_attention(a, kv, o, n_heads, scale, hs);
  if (st != DV_OK) return st;
  AxpyArgs ax{};
  ax.d = a->d; ax.nrows = n_heads * a->dh; ax.M = a->WoT; ax.m_rows = a->H * a->dh; ax.set = o.heads;
  ax.dh = a->dh; ax.coef = nullptr; ax.part = o.part; ax.n_split = attn_nsplit(a, kv, n_heads);
  ax.resid = nullptr; ax.bias = a->bo; ax.out = out; ax.out2 = nullptr; ax.partial = o.axp; ax.cnt = o.axc;
  return enqueue_axpy("oproj", a->wtype, ax, hs);
}

// ------------------------------------------------------------ 4-bit sparse MLP
static dv_status check_mlp_q4(const dv_mlp_q4* m) {
  if (m == nullptr || m->W1T == nullptr || m->W2T == nullptr || m->S1 == nullptr || m->S2 == nullptr)
    return DV_ERR_NULL;
  if (m->act != DV_ACT_RELU && m->act != DV_ACT_GELU) return DV_ERR_ARG;
  if (m->reserved != 0) return DV_ERR_ARG;
  if (m->d <= 0 || m->n <= 0) return DV_ERR_SHAPE;
  if (m->d % 32 != 0 || !aligned16(m->W1T) || !aligned16(m->W2T)) return DV_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(m->S1) & 1u) || (reinterpret_cast<uintptr_t>(m->S2) & 1u)) return DV_ERR_ALIGN;
  if (m->d > kMaxWidth) return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

extern "C" size_t dv_sparse_mlp_q4_workspace_bytes(const dv_mlp_q4* m, int32_t n_idx) {
  if (m == nullptr || m->d <= 0 || m->n <= 0 || n_idx < 0) return 0;
  Workspace w(nullptr);
  w.take<float>((size_t)n_idx * sizeof(float));
  w.take<float>(axpy_partial_bytes(m->d));
  w.take<uint32_t>(kAxpyMaxSpans * sizeof(uint32_t));
  w.take<int32_t>(sizeof(int32_t));
  return w.off;
}

extern "C" dv_status dv_sparse_mlp_q4(const dv_mlp_q4* m, const float* x, const int32_t* idx, int32_t n_idx,
                                      float* out, void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_mlp_q4(m);
  if (st != DV_OK) return st;
  if (x == nullptr || out == nullptr || (idx == nullptr && n_idx > 0)) return DV_ERR_NULL;
  if (n_idx < 0 || n_idx > m->n) return DV_ERR_SHAPE;
  if (!aligned16(x) || !aligned16(out)) return DV_ERR_ALIGN;
  if ((m->b1 != nullptr && !aligned16(m->b1)) || (m->b2 != nullptr && !aligned16(m->b2))) return DV_ERR_ALIGN;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  if (dv_sparse_mlp_q4_workspace_bytes(m, n_idx) > ws_bytes) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  Workspace w(ws);
  float* h = w.take<float>((size_t)n_idx * sizeof(float));
  float* axp = w.take<float>(axpy_partial_bytes(m->d));
  uint32_t* axc = w.take<uint32_t>(kAxpyMaxSpans * sizeof(uint32_t));
  int32_t* flag = w.take<int32_t>(sizeof(int32_t));
  if (flags & DV_VALIDATE) {
    st = validate_sets(idx, 1, n_idx, m->n, flag, hs);
    if (st != DV_OK) return st;
  }
  Fc1Args f{};
  f.d = m->d; f.k = n_idx; f.n = m->n; f.x = x; f.W1T = m->W1T; f.b1 = m->b1; f.set = idx;
  f.s1 = static_cast<const _Float16*>(m->S1); f.act = m->act; f.h = h; f.clear = axc; f.clear_n = kAxpyMaxSpans;
  DV_LAUNCH("fc1", hs, launch_fc1(DV_Q4, f, hs));
  AxpyArgs ax{};
  ax.d = m->d; ax.nrows = n_idx; ax.M = m->W2T; ax.m_rows = m->n; ax.set = idx; ax.dh = 0; ax.coef = h;
  ax.scales = static_cast<const _Float16*>(m->S2); ax.bias = m->b2; ax.out = out; ax.partial = axp; ax.cnt = axc;
  return enqueue_axpy("fc2", DV_Q4, ax, hs);
}

// ------------------------------------------- sparse attention, missing keys and values
static constexpr int kMaxFillPos = 32768;   // the fill launch lists missing positions in LDS

extern "C" dv_status dv_sparse_attn_kvfill(const dv_attn* a, const float* x, const dv_kv* kv, void* Y,
                                           uint8_t* valid, const int32_t* heads, int32_t n_heads, float scale,
                                           float* out, void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_attn(a);
  if (st != DV_OK) return st;
  if (x == nullptr || out == nullptr || Y == nullptr || valid == nullptr || (heads == nullptr && n_heads > 0))
    return DV_ERR_NULL;
  if (n_heads < 0 || n_heads > a->H) return DV_ERR_SHAPE;
  if ((st = check_kv(kv, a, 1)) != DV_OK) return st;
  if (!aligned16(x) || !aligned16(out) || !aligned16(Y)) return DV_ERR_ALIGN;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (!isfinite(scale)) return DV_ERR_ARG;
  if (a->bo != nullptr && !aligned16(a->bo)) return DV_ERR_ALIGN;
  if (kv->pos[0] > kMaxFillPos) return DV_ERR_UNSUPPORTED;
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  Workspace w(ws);
  AttnWs o;
  if (attn_ws_layout(a, 1, n_heads, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  if (flags & DV_VALIDATE) {
    st = validate_sets(heads, 1, n_heads, a->H, o.flag, hs);
    if (st != DV_OK) return st;
  }
  const int pos = kv->pos[0];
  KvFillArgs f{};
  f.d = a->d; f.H = a->H; f.dh = a->dh; f.cap = kv->cap; f.pos = pos; f.n_heads = n_heads;
  f.x = x; f.Y = Y; f.valid = valid; f.heads = heads;
  f.Wk = a->Wk; f.Wv = a->Wv; f.bk = a->bk; f.bv = a->bv; f.K = kv->K; f.V = kv->V;
  // The missing positions are listed by a workgroup hosted in the QKV launch, into the
  // row-axpy partial buffer of the workspace (unused until the out-projection), when they
  // fit; the fill then runs after QKV. Otherwise every fill workgroup lists its head's
  // positions itself, in a fill before QKV.
  const int stride = max(pos, 1);
  const bool listed =
      n_heads > 0 && (size_t)n_heads * (stride + 1) <= axpy_partial_bytes(a->d) / sizeof(int32_t);
  int32_t* list = listed ? reinterpret_cast<int32_t*>(o.axp) : nullptr;
  if (n_heads > 0 && !listed) {
    DV_LAUNCH("kv_fill", hs, launch_kv_fill(a->wtype, kv->ktype, f, hs));
  } else if (n_heads == 0) {   // no head selected: nothing to compute, the input is still kept
    DV_LAUNCH("kv_keep", hs, launch_keep_input(kv->ktype, f, hs));
  }
  QkvArgs q{};
  q.d = a->d; q.H = a->H; q.dh = a->dh; q.cap = kv->cap; q.pos = pos; q.n_heads = n_heads;
  q.x = x;
  q.Wq = a->Wq; q.Wk = a->Wk; q.Wv = a->Wv; q.bq = a->bq; q.bk = a->bk; q.bv = a->bv;
  q.K = kv->K; q.V = kv->V; q.q = o.q; q.heads_in = heads; q.heads_ws = o.heads;
  q.clear = o.axc; q.clear_n = kAxpyMaxSpans; q.valid = valid;
  if (listed) {
    q.list = list; q.list_stride = stride; q.list_count = list + (size_t)n_heads * stride;
  }
  DV_LAUNCH("qkv", hs, launch_qkv(a->wtype, kv->ktype, q, hs));   // also marks row pos of every head
  if (listed) DV_LAUNCH("kv_fill", hs, launch_kv_fill_listed(a->wtype, kv->ktype, f, list, stride, hs));
  if (n_heads == 0) {
    AxpyArgs ax{};
    ax.d = a->d; ax.nrows = 0; ax.M = a->WoT; ax.m_rows = a->H * a->dh; ax.set = o.heads; ax.dh = 0;
    ax.coef = o.q; ax.bias = a->bo; ax.out = out;
    DV_LAUNCH("oproj", hs, launch_axpy(a->wtype, ax, hs));
    return DV_OK;
  }
  if ((st = enqueue_attention(a, kv, o, n_heads, scale, hs, valid)) != DV_OK) return st;
  AxpyArgs ax{};
  ax.d = a->d; ax.nrows = n_heads * a->dh; ax.M = a->WoT; ax.m_rows = a->H * a->dh; ax.set = o.heads;
  ax.dh = a->dh; ax.coef = nullptr; ax.part = o.part; ax.n_split = attn_nsplit(a, kv, n_heads);
  ax.resid = nullptr; ax.bias = a->bo; ax.out = out; ax.out2 = nullptr; ax.partial = o.axp; ax.cnt = o.axc;
  return enqueue_axpy("oproj", a->wtype, ax, hs);
}

// ------------------------------------------------------------- decoder layer
struct BlockWs {
  float* hid_h; float* hid_m; float* s_h; float* s_m; int32_t* heads; int32_t* idx;
  float* q; float* part; float* ytilde; float* xhat; float* h; float* axp; uint32_t* axc; int32_t* flag;
};

static size_t block_ws_layout(const dv_attn* a, const dv_predictor* pa, const dv_predictor* pm, int B, int kh,
                              int km, Workspace& w, BlockWs* o) {
  o->hid_h = w.take<float>((size_t)B * pa->r * sizeof(float));
  o->hid_m = w.take<float>((size_t)B * pm->r * sizeof(float));
  o->s_h = w.take<float>((size_t)B * pa->n_out * sizeof(float));
  o->s_m = w.take<float>((size_t)B * pm->n_out * sizeof(float));
  o->heads = w.take<int32_t>((size_t)B * kh * sizeof(int32_t));
  o->idx = w.take<int32_t>((size_t)B * km * sizeof(int32_t));
  o->q = w.take<float>((size_t)B * kh * a->dh * sizeof(float));
  o->part = w.take<float>((size_t)B * kh * kAttnMaxSplit * (a->dh + 2) * sizeof(float));
  o->ytilde = w.take<float>((size_t)B * a->d * sizeof(float));
  o->xhat = w.take<float>((size_t)B * a->d * sizeof(float));
  o->h = w.take<float>((size_t)B * km * sizeof(float));
  o->axp = w.take<float>(axpy_partial_bytes(a->d));
  o->axc = w.take<uint32_t>(2 * kAxpyMaxSpans * sizeof(uint32_t));   // out-projection, fc2
  o->flag = w.take<int32_t>(sizeof(int32_t));
  return w.off;
}

extern "C" size_t dv_sparse_block_workspace_bytes(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa,
                                                  const dv_predictor* pm, const dv_kv* kv, int32_t B,
                                                  int32_t k_heads, int32_t k_mlp) {
  if (a == nullptr || m == nullptr || pa == nullptr || pm == nullptr || kv == nullptr || B <= 0 ||
      k_heads < 0 || k_mlp < 0 || a->d <= 0 || a->dh <= 0 || kv->cap <= 0 || pa->r <= 0 || pm->r <= 0 ||
      pa->n_out <= 0 || pm->n_out <= 0 || !dtype_ok(a->wtype) || !dtype_ok(m->wtype))
    return 0;
  if (B > 1) return batch_block_ws(a, m, pa, pm, B, k_heads, k_mlp);
  Workspace w(nullptr);
  BlockWs o;
  return block_ws_layout(a, pa, pm, B, k_heads, k_mlp, w, &o);
}

dv_status dv::check_predictor_for(const dv_predictor* p, int d, int n_out) {
  if (p == nullptr || p->AT == nullptr || p->BT == nullptr) return DV_ERR_NULL;
  if (!dtype_ok(p->wtype)) return DV_ERR_DTYPE;
  if (p->d != d || p->n_out != n_out || p->r <= 0) return DV_ERR_SHAPE;
  if (p->d % chunk_elems(p->wtype) != 0 || p->r % chunk_elems(p->wtype) != 0) return DV_ERR_ALIGN;
  if (!aligned16(p->AT) || !aligned16(p->BT)) return DV_ERR_ALIGN;
  if (p->r > kMaxWidth) return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

extern "C" dv_status dv_sparse_block(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa,
                                     const dv_predictor* pm, const dv_ln* ln, const dv_kv* kv,
                                     const float* x_in, float* x_out, int32_t B, int32_t k_heads,
                                     int32_t k_mlp, int32_t mode, int32_t batch_mode, float scale,
                                     int32_t* heads_out, int32_t* idx_out, void* ws, size_t ws_bytes,
                                     uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_attn(a);
  if (st != DV_OK) return st;
  if ((st = check_mlp(m)) != DV_OK) return st;
  if (m->d != a->d) return DV_ERR_SHAPE;
  if ((st = check_predictor_for(pa, a->d, a->H)) != DV_OK) return st;
  if ((st = check_predictor_for(pm, a->d, m->n)) != DV_OK) return st;
  if (pa->wtype != pm->wtype) return DV_ERR_DTYPE;
  if (x_in == nullptr || x_out == nullptr) return DV_ERR_NULL;
  if (B <= 0) return DV_ERR_SHAPE;
  if ((st = check_kv(kv, a, B)) != DV_OK) return st;
  if ((st = check_ln(ln)) != DV_OK) return st;
  if (k_heads < 1 || k_heads > a->H || k_mlp < 1 || k_mlp > m->n) return DV_ERR_SHAPE;
  if (a->H > 512) return DV_ERR_UNSUPPORTED;
  if (mode != DV_LOOKAHEAD && mode != DV_SEQUENTIAL) return DV_ERR_ARG;
  if (batch_mode != DV_MLP_UNION && batch_mode != DV_MLP_MASKED) return DV_ERR_ARG;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (!isfinite(scale)) return DV_ERR_ARG;
  if (!aligned16(x_in) || !aligned16(x_out)) return DV_ERR_ALIGN;
  if ((a->bo && !aligned16(a->bo)) || (m->b2 && !aligned16(m->b2))) return DV_ERR_ALIGN;
  if (B > 1) {
    if (!batch_ok(B, a->wtype) || m->wtype != DV_F16 || pa->wtype != DV_F16 || m->n > kMaxUnionN ||
        pa->r > batch_max_rank(B) || pm->r > batch_max_rank(B))
      return DV_ERR_UNSUPPORTED;
    if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
    return batch_block(a, m, pa, pm, ln, kv, x_in, x_out, B, k_heads, k_mlp, mode, batch_mode, scale, heads_out,
                       idx_out, ws, ws_bytes, static_cast<hipStream_t>(stream));
  }
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  Workspace w(ws);
  BlockWs o;
  if (block_ws_layout(a, pa, pm, B, k_heads, k_mlp, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);

  const float* g1 = ln ? ln->g1 : nullptr;
  const float* be1 = ln ? ln->be1 : nullptr;
  const float* g2 = ln ? ln->g2 : nullptr;
  const float* be2 = ln ? ln->be2 : nullptr;
  const float eps = ln ? ln->eps : 0.f;
  const bool ahead = mode == DV_LOOKAHEAD;

  // 1. Predictor hidden layers from LN1(y) (both in look-ahead mode).
  PredHidArgs ha{};
  ha.d = a->d; ha.B = 1; ha.x = x_in; ha.g = g1; ha.be = be1; ha.eps = eps;
  ha.AT0 = pa->AT; ha.r0 = pa->r; ha.hid0 = o.hid_h;
  ha.AT1 = ahead ? pm->AT : nullptr; ha.r1 = ahead ? pm->r : 0; ha.hid1 = o.hid_m;
  ha.xhat_out = o.xhat;   // LN1(y), reused by the QKV launch
  DV_LAUNCH("pred_hidden", hs, launch_pred_hidden(pa->wtype, ha, hs));
  // 2. Predictor scores.
  PredScoreArgs sa{};
  sa.r0 = pa->r; sa.n0 = a->H; sa.BT0 = pa->BT; sa.hid0 = o.hid_h; sa.s0 = o.s_h;
  sa.r1 = ahead ? pm->r : 0; sa.n1 = ahead ? m->n : 0; sa.BT1 = pm->BT; sa.hid1 = o.hid_m; sa.s1 = o.s_m;
  sa.B = 1;
  // The head set is selected by workgroup 0 of this launch when a head-predictor row
  // is at most 128 chunks (two wavefront loads); otherwise by a launch of its own.
  const bool host_heads = pa->r / chunk_elems(pa->wtype) <= 128;
  if (host_heads) {
    sa.sel_k0 = k_heads; sa.sel_set0 = o.heads; sa.sel_set0_out = heads_out;
  }
  DV_LAUNCH("pred_scores", hs, launch_pred_scores(pa->wtype, sa, hs));
  if (!host_heads)
    DV_LAUNCH("select_heads", hs,
              launch_select(o.s_h, 1, a->H, DV_SELECT_TOPK, k_heads, 0.f, o.heads, k_heads, nullptr, heads_out, hs));
  // 3. Gathered QKV of the selected heads + cache append.
  QkvArgs q{};
  q.d = a->d; q.H = a->H; q.dh = a->dh; q.cap = kv->cap; q.pos = kv->pos[0]; q.n_heads = k_heads;
  q.x = o.xhat;
  q.Wq = a->Wq; q.Wk = a->Wk; q.Wv = a->Wv; q.bq = a->bq; q.bk = a->bk; q.bv = a->bv;
  q.K = kv->K; q.V = kv->V; q.q = o.q; q.heads_in = o.heads; q.heads_ws = nullptr;
  q.clear = o.axc; q.clear_n = kAxpyMaxSpans;
  if (ahead) {
    // the neuron selection (from the LN1(y) scores) runs in one extra workgroup of
    // the QKV launch, beside its weight stream, off the critical path (Section 4.3)
    q.sel_n = m->n; q.sel_scores = o.s_m; q.sel_k = k_mlp; q.sel_idx = o.idx; q.sel_idx_out = idx_out;
  }
  DV_LAUNCH("qkv", hs, launch_qkv(a->wtype, kv->ktype, q, hs));
  // 4. Split-KV attention.
  AttnWs ao{};
  ao.heads = o.heads; ao.q = o.q; ao.part = o.part;
  if ((st = enqueue_attention(a, kv, ao, k_heads, scale, hs)) != DV_OK) return st;
  // 5. Out-projection + residual: y~ = y + MHA(LN1(y)).
  AxpyArgs ax{};
  ax.d = a->d; ax.nrows = k_heads * a->dh; ax.M = a->WoT; ax.m_rows = a->H * a->dh; ax.set = o.heads;
  ax.dh = a->dh; ax.coef = nullptr; ax.part = o.part; ax.n_split = attn_nsplit(a, kv, k_heads);
  ax.resid = x_in; ax.bias = a->bo; ax.out = o.ytilde; ax.out2 = nullptr; ax.partial = o.axp; ax.cnt = o.axc;
  if ((st = enqueue_axpy("oproj", a->wtype, ax, hs)) != DV_OK) return st;
  // 5b. Sequential mode: the neuron predictor reads LN2(y~).
  if (!ahead) {
    PredHidArgs hm{};
    hm.d = a->d; hm.B = 1; hm.x = o.ytilde; hm.g = g2; hm.be = be2; hm.eps = eps;
    hm.AT0 = pm->AT; hm.r0 = pm->r; hm.hid0 = o.hid_m; hm.r1 = 0;
    DV_LAUNCH("pred_hidden_mlp", hs, launch_pred_hidden(pm->wtype, hm, hs));
    PredScoreArgs sm{};
    sm.r0 = pm->r; sm.n0 = m->n; sm.BT0 = pm->BT; sm.hid0 = o.hid_m; sm.s0 = o.s_m; sm.n1 = 0; sm.B = 1;
    DV_LAUNCH("pred_scores_mlp", hs, launch_pred_scores(pm->wtype, sm, hs));
    DV_LAUNCH("select_mlp", hs,
              launch_select(o.s_m, 1, m->n, DV_SELECT_TOPK, k_mlp, 0.f, o.idx, k_mlp, nullptr, idx_out, hs));
  }
  // 6. fc1 + ReLU on LN2(y~).
  Fc1Args f{};
  f.d = m->d; f.k = k_mlp; f.n = m->n; f.x = o.ytilde; f.g = g2; f.be = be2; f.eps = eps;
  f.W1T = m->W1T; f.b1 = m->b1; f.set = o.idx; f.h = o.h; f.act = m->act;
  f.clear = o.axc + kAxpyMaxSpans; f.clear_n = kAxpyMaxSpans;
  DV_LAUNCH("fc1", hs, launch_fc1(m->wtype, f, hs));
  // 7. fc2 + residual: y^ = y~ + MLP(LN2(y~)).
  AxpyArgs ay{};
  ay.d = m->d; ay.nrows = k_mlp; ay.M = m->W2T; ay.m_rows = m->n; ay.set = o.idx; ay.dh = 0;
  ay.coef = o.h; ay.resid = o.ytilde; ay.bias = m->b2; ay.out = x_out; ay.out2 = nullptr; ay.partial = o.axp;
  ay.cnt = o.axc + kAxpyMaxSpans;
  if ((st = enqueue_axpy("fc2", m->wtype, ay, hs)) != DV_OK) return st;
  return DV_OK;
}

// -------------------------------------------------------------------- misc
extern "C" const char* dv_status_string(int32_t s) {
  switch (s) {
    case DV_OK: return "ok";
    case DV_ERR_NULL: return "a required pointer is NULL";
    case DV_ERR_SHAPE: return "inconsistent or out-of-range sizes";
    case DV_ERR_DTYPE: return "unknown or mismatched dtype";
    case DV_ERR_ALIGN: return "pointer or row not 16-byte aligned";
    case DV_ERR_WORKSPACE: return "workspace NULL, too small or not 256-byte aligned";
    case DV_ERR_INDEX: return "index set not strictly ascending within range";
    case DV_ERR_HIP: return "HIP runtime or launch failure";
    case DV_ERR_UNSUPPORTED: return "valid request not supported by this build";
    case DV_ERR_ARG: return "invalid mode or flag";
    default: return "unknown status";
  }
}

extern "C" int32_t dv_abi_version(void) { return DV_ABI_VERSION; }
