// dv_sparse_decode: several decoder layers for one token with the cross-layer
// look-ahead of Section 4.3 ("Approach"): the sets that layer l+1 uses are predicted
// from layer l's normalised input x_l = LN1^l(y_l), so the prediction needs nothing
// that layer l computes and is folded into layer l's own launches instead of running
// as launches of its own between layers:
//   QKV(l)    the Q/K/V rows of S_A^l and, over the same staged x_l, the first-layer
//             rows of layer l+1's two predictors (one HBM pass, one launch); one extra
//             workgroup selects S_M^l from the neuron scores computed during layer l-1
//   attn(l)   split-KV attention
//   scores    layer l+1's predictor scores; the head set S_A^{l+1} in workgroup 0
//   oproj(l), fc1(l) (LN2 in the launch, S_M^l), fc2(l) -> y_{l+1}
// Layer 0's head set and neuron scores come from a prologue on LN1^0(y_0). Every
// launch goes to one stream; the head sets are double buffered (attention and
// out-projection of layer l read S_A^l while layer l+1's set is written), the neuron
// scores, the neuron set and the predictor hidden vectors are consumed before they
// are rewritten.
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

namespace {
struct DecodeWs {
  float *hid_h, *hid_m, *s_h, *s_m;    // predictors: hidden vectors, scores
  int32_t *heads[2], *idx;             // head sets (double buffered), neuron set
  float *q, *part, *ytilde, *h, *axp;  // the layer's own intermediates
  uint32_t* axc;
  float* y[2];                         // layer outputs, ping-pong
};

size_t decode_ws_layout(const dv_layer* L0, int kh, int km, Workspace& w, DecodeWs* o) {
  const dv_attn& a = L0->attn;
  o->hid_h = w.take<float>((size_t)L0->pa.r * 4);
  o->hid_m = w.take<float>((size_t)L0->pm.r * 4);
  o->s_h = w.take<float>((size_t)a.H * 4);
  o->s_m = w.take<float>((size_t)L0->mlp.n * 4);
  for (int i = 0; i < 2; ++i) o->heads[i] = w.take<int32_t>((size_t)kh * 4);
  o->idx = w.take<int32_t>((size_t)km * 4);
  o->q = w.take<float>((size_t)kh * a.dh * 4);
  o->part = w.take<float>((size_t)kh * kAttnMaxSplit * (a.dh + 2) * 4);
  o->ytilde = w.take<float>((size_t)a.d * 4);
  o->h = w.take<float>((size_t)km * 4);
  o->axp = w.take<float>(axpy_partial_bytes(a.d));
  o->axc = w.take<uint32_t>(2 * kAxpyMaxSpans * 4);
  for (int i = 0; i < 2; ++i) o->y[i] = w.take<float>((size_t)a.d * 4);
  return w.off;
}

// Every layer must have the shapes and types of layer 0 (one workspace layout serves all).
bool same_shape(const dv_layer& a, const dv_layer& b) {
  return a.attn.d == b.attn.d && a.attn.H == b.attn.H && a.attn.dh == b.attn.dh && a.attn.wtype == b.attn.wtype &&
         a.mlp.d == b.mlp.d && a.mlp.n == b.mlp.n && a.mlp.wtype == b.mlp.wtype && a.pa.r == b.pa.r &&
         a.pm.r == b.pm.r && a.pa.wtype == b.pa.wtype && a.pm.wtype == b.pm.wtype && a.kv.ktype == b.kv.ktype;
}

dv_status check_layer(const dv_layer& L, int kh, int km) {
  dv_status st;
  if ((st = check_attn(&L.attn)) != DV_OK) return st;
  if ((st = check_mlp(&L.mlp)) != DV_OK) return st;
  if (L.mlp.d != L.attn.d) return DV_ERR_SHAPE;
  if ((st = check_predictor_for(&L.pa, L.attn.d, L.attn.H)) != DV_OK) return st;
  if ((st = check_predictor_for(&L.pm, L.attn.d, L.mlp.n)) != DV_OK) return st;
  if (L.pa.wtype != L.pm.wtype) return DV_ERR_DTYPE;
  if ((st = check_kv(&L.kv, &L.attn, 1)) != DV_OK) return st;
  if ((st = check_ln(&L.ln)) != DV_OK) return st;
  if (kh < 1 || kh > L.attn.H || km < 1 || km > L.mlp.n) return DV_ERR_SHAPE;
  if (L.attn.H > 512) return DV_ERR_UNSUPPORTED;
  if ((L.attn.bo && !aligned16(L.attn.bo)) || (L.mlp.b2 && !aligned16(L.mlp.b2))) return DV_ERR_ALIGN;
  return DV_OK;
}

// First layer of layer j's two predictors on LN(x) (layer norm g, be): a launch of its
// own (the prologue, or when the predictor and Q/K/V weights differ in type).
dv_status enqueue_pred_hidden(const dv_layer& Lj, const float* x, const float* g, const float* be, float eps,
                              const DecodeWs& o, hipStream_t st) {
  PredHidArgs ha{};
  ha.d = Lj.attn.d; ha.B = 1; ha.x = x; ha.g = g; ha.be = be; ha.eps = eps;
  ha.AT0 = Lj.pa.AT; ha.r0 = Lj.pa.r; ha.hid0 = o.hid_h;
  ha.AT1 = Lj.pm.AT; ha.r1 = Lj.pm.r; ha.hid1 = o.hid_m;
  DV_LAUNCH("pred_hidden", st, launch_pred_hidden(Lj.pa.wtype, ha, st));
  return DV_OK;
}

// Second layer of layer j's predictors: neuron scores s_m, head scores and the head set
// (selected in workgroup 0 of the launch when a head-predictor row is short).
dv_status enqueue_pred_scores(const dv_layer& Lj, int kh, const DecodeWs& o, int32_t* heads, int32_t* heads_out,
                              hipStream_t st) {
  PredScoreArgs sa{};
  sa.r0 = Lj.pa.r; sa.n0 = Lj.attn.H; sa.BT0 = Lj.pa.BT; sa.hid0 = o.hid_h; sa.s0 = o.s_h;
  sa.r1 = Lj.pm.r; sa.n1 = Lj.mlp.n; sa.BT1 = Lj.pm.BT; sa.hid1 = o.hid_m; sa.s1 = o.s_m;
  sa.B = 1;
  const bool host_heads = Lj.pa.r / chunk_elems(Lj.pa.wtype) <= 128;
  if (host_heads) {
    sa.sel_k0 = kh; sa.sel_set0 = heads; sa.sel_set0_out = heads_out;
  }
  DV_LAUNCH("pred_scores", st, launch_pred_scores(Lj.pa.wtype, sa, st));
  if (!host_heads)
    DV_LAUNCH("select_heads", st,
              launch_select(o.s_h, 1, Lj.attn.H, DV_SELECT_TOPK, kh, 0.f, heads, kh, nullptr, heads_out, st));
  return DV_OK;
}

// Layer l's sparse block on the head set `heads` (the neuron set is selected in the QKV
// launch from the scores o.s_m): y_out = y~ + MLP(LN2(y~)), y~ = y + MHA(LN1(y)). With
// `next`, layer l+1's predictors run on LN1(y) inside the launches (see the top).
dv_status enqueue_layer(const dv_layer& L, const dv_layer* next, const float* y, float* y_out, int kh, int km,
                        float scale, const int32_t* heads, int32_t* idx_out, int32_t* next_heads,
                        int32_t* next_heads_out, const DecodeWs& o, hipStream_t st) {
  const dv_attn& a = L.attn;
  const dv_mlp& m = L.mlp;
  const int pos = L.kv.pos[0];
  const bool fold = next != nullptr && next->pa.wtype == a.wtype;   // predictor rows in the QKV launch
  QkvArgs q{};
  q.d = a.d; q.H = a.H; q.dh = a.dh; q.cap = L.kv.cap; q.pos = pos; q.n_heads = kh;
  q.x = y; q.g = L.ln.g1; q.be = L.ln.be1; q.eps = L.ln.eps;
  q.Wq = a.Wq; q.Wk = a.Wk; q.Wv = a.Wv; q.bq = a.bq; q.bk = a.bk; q.bv = a.bv;
  q.K = L.kv.K; q.V = L.kv.V; q.q = o.q; q.heads_in = heads; q.heads_ws = nullptr;
  q.clear = o.axc; q.clear_n = kAxpyMaxSpans;
  q.sel_n = m.n; q.sel_scores = o.s_m; q.sel_k = km; q.sel_idx = o.idx; q.sel_idx_out = idx_out;
  if (fold) {
    q.AT0 = next->pa.AT; q.r0 = next->pa.r; q.hid0 = o.hid_h;
    q.AT1 = next->pm.AT; q.r1 = next->pm.r; q.hid1 = o.hid_m;
  }
  DV_LAUNCH("qkv", st, launch_qkv(a.wtype, L.kv.ktype, q, st));
  dv_status s;
  if (next != nullptr && !fold &&
      (s = enqueue_pred_hidden(*next, y, L.ln.g1, L.ln.be1, L.ln.eps, o, st)) != DV_OK)
    return s;
  AttnArgs at{};
  at.H = a.H; at.dh = a.dh; at.cap = L.kv.cap; at.posb[0] = pos; at.n_heads = kh;
  at.chunk = attn_chunk(kh, pos + 1, a.dh, L.kv.ktype);
  at.n_split = (pos + 1 + at.chunk - 1) / at.chunk;
  at.q = o.q; at.heads = heads; at.K = L.kv.K; at.V = L.kv.V; at.scale = scale; at.part = o.part;
  DV_LAUNCH("attn", st, launch_attn(L.kv.ktype, at, 1, st));
  if (next != nullptr && (s = enqueue_pred_scores(*next, kh, o, next_heads, next_heads_out, st)) != DV_OK) return s;
  AxpyArgs ax{};
  ax.d = a.d; ax.nrows = kh * a.dh; ax.M = a.WoT; ax.m_rows = a.H * a.dh; ax.set = heads;
  ax.dh = a.dh; ax.coef = nullptr; ax.part = o.part; ax.n_split = at.n_split;
  ax.resid = y; ax.bias = a.bo; ax.out = o.ytilde; ax.out2 = nullptr; ax.partial = o.axp; ax.cnt = o.axc;
  DV_LAUNCH("oproj", st, launch_axpy(a.wtype, ax, st));
  Fc1Args f{};
  f.d = m.d; f.k = km; f.n = m.n; f.x = o.ytilde; f.g = L.ln.g2; f.be = L.ln.be2; f.eps = L.ln.eps;
  f.W1T = m.W1T; f.b1 = m.b1; f.set = o.idx; f.h = o.h; f.act = m.act;
  f.clear = o.axc + kAxpyMaxSpans; f.clear_n = kAxpyMaxSpans;
  DV_LAUNCH("fc1", st, launch_fc1(m.wtype, f, st));
  AxpyArgs ay{};
  ay.d = m.d; ay.nrows = km; ay.M = m.W2T; ay.m_rows = m.n; ay.set = o.idx; ay.dh = 0;
  ay.coef = o.h; ay.resid = o.ytilde; ay.bias = m.b2; ay.out = y_out; ay.out2 = nullptr; ay.partial = o.axp;
  ay.cnt = o.axc + kAxpyMaxSpans;
  DV_LAUNCH("fc2", st, launch_axpy(m.wtype, ay, st));
  return DV_OK;
}
}  // namespace

}  // namespace dv

using namespace dv;

extern "C" size_t dv_sparse_decode_workspace_bytes(const dv_layer* layers, int32_t n_layers, int32_t k_heads,
                                                   int32_t k_mlp) {
  if (layers == nullptr || n_layers <= 0 || k_heads < 0 || k_mlp < 0) return 0;
  const dv_layer& L0 = layers[0];
  if (L0.attn.d <= 0 || L0.attn.dh <= 0 || L0.attn.H <= 0 || L0.mlp.n <= 0 || L0.pa.r <= 0 || L0.pm.r <= 0)
    return 0;
  Workspace w(nullptr);
  DecodeWs o;
  return decode_ws_layout(&L0, k_heads, k_mlp, w, &o);
}

extern "C" dv_status dv_sparse_decode(const dv_layer* layers, int32_t n_layers, const float* x_in, float* x_out,
                                      int32_t k_heads, int32_t k_mlp, float scale, int32_t* heads_out,
                                      int32_t* idx_out, void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  if (layers == nullptr || x_in == nullptr || x_out == nullptr) return DV_ERR_NULL;
  if (n_layers <= 0) return DV_ERR_SHAPE;
  dv_status st;
  for (int l = 0; l < n_layers; ++l) {
    if ((st = check_layer(layers[l], k_heads, k_mlp)) != DV_OK) return st;
    if (!same_shape(layers[l], layers[0])) return DV_ERR_SHAPE;
  }
  if (!aligned16(x_in) || !aligned16(x_out)) return DV_ERR_ALIGN;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (!isfinite(scale)) return DV_ERR_ARG;
  if (!ws_ok(ws)) return DV_ERR_WORKSPACE;
  Workspace w(ws);
  DecodeWs o;
  if (decode_ws_layout(&layers[0], k_heads, k_mlp, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  auto y_of = [&](int l) -> float* {
    return l == 0 ? const_cast<float*>(x_in) : (l == n_layers ? x_out : o.y[(l - 1) & 1]);
  };
  auto hout = [&](int j) { return heads_out ? heads_out + (size_t)j * k_heads : nullptr; };
  auto iout = [&](int j) { return idx_out ? idx_out + (size_t)j * k_mlp : nullptr; };
  // prologue: layer 0's predictors on LN1^0(y_0)
  const dv_layer& L0 = layers[0];
  if ((st = enqueue_pred_hidden(L0, x_in, L0.ln.g1, L0.ln.be1, L0.ln.eps, o, hs)) != DV_OK) return st;
  if ((st = enqueue_pred_scores(L0, k_heads, o, o.heads[0], hout(0), hs)) != DV_OK) return st;
  for (int l = 0; l < n_layers; ++l) {
    const dv_layer* next = l + 1 < n_layers ? &layers[l + 1] : nullptr;
    if ((st = enqueue_layer(layers[l], next, y_of(l), y_of(l + 1), k_heads, k_mlp, scale, o.heads[l & 1], iout(l),
                            o.heads[(l + 1) & 1], hout(l + 1), o, hs)) != DV_OK)
      return st;
  }
  return DV_OK;
}
