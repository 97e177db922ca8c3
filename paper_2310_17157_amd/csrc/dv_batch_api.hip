// Host side of the batched path (1 < B <= 32): workspace layouts and launch sequences
// of the sparsified MLP, the sparsified attention and the decoder layer on the matrix
// cores. Arguments arrive validated by the C ABI entry points.
//
// Sparsified MLP (Eq. (1)) over the union U of the batch's neuron sets (Section 5.2):
//   [union] -> x-hat fp16 -> fc1 on U (MFMA, K-split partials) -> ReLU/bias/mask
//   -> fc2 on U (MFMA, row-split partials) -> sum + b2 (+ residual).
// Sparsified attention (Eq. (2)) with a head set per sequence: the union of the head
// sets gives the Q/K/V rows read once for the batch; each (sequence, head) pair keeps
// its own query, cache rows and attention; the out-projection contracts over the
// union's W^O rows with zero coefficients for heads a sequence did not select.
#include <math.h>

#include <algorithm>

#include "dv_internal.hpp"

namespace dv {

static int round_up(int v, int m) { return (v + m - 1) / m * m; }

int batch_nb(int B) { return B <= 16 ? 16 : 32; }

// ---------------------------------------------------------------- MLP
struct BMlp {
  _Float16* X16; int32_t* U; int32_t* cnt; uint32_t* mask; float* P; _Float16* C;
  float* P2;
  int Kpad, S, Ks, umax, nrows_pad, ldc, S2;
};

static size_t bmlp_layout(int d, int n, int B, int n_idx, bool per_seq, Workspace& w, BMlp* o) {
  const int NB = batch_nb(B);
  o->Kpad = round_up(d, 32);
  mrows_split(o->Kpad, NB, &o->S, &o->Ks);
  o->umax = per_seq ? (int)std::min<long>(n, (long)B * n_idx) : n_idx;
  o->nrows_pad = round_up(std::max(o->umax, 1), 16);
  o->ldc = round_up(std::max(o->umax, 1), 64);
  o->S2 = mcols_split(d, o->umax);
  o->X16 = w.take<_Float16>((size_t)NB * o->Kpad * 2);
  o->U = w.take<int32_t>(per_seq ? (size_t)o->umax * 4 : 0);
  o->cnt = w.take<int32_t>(4);
  o->mask = w.take<uint32_t>(per_seq ? (size_t)o->umax * 4 : 0);
  o->P = w.take<float>((size_t)o->S * o->nrows_pad * NB * 4);
  o->C = w.take<_Float16>((size_t)NB * o->ldc * 2);
  o->P2 = w.take<float>((size_t)o->S2 * B * d * 4);
  return w.off;
}

size_t batch_mlp_ws(const dv_mlp* m, int B, int n_idx, int per_seq) {
  Workspace w(nullptr);
  BMlp o;
  return bmlp_layout(m->d, m->n, B, n_idx, per_seq != 0, w, &o);
}

// The MLP on x16 (already normalised, fp16 [NB][Kpad]) for the sets `idx`.
// union_done: the union (and masks) were built by the launch that cast x.
static dv_status bmlp_run(const dv_mlp* m, const BMlp& o, int B, const int32_t* idx, int n_idx, bool per_seq,
                          bool masked, const float* resid, float* out, hipStream_t hs, bool union_done = false) {
  const int NB = batch_nb(B);
  const int32_t* list = idx;
  const int32_t* list_count = nullptr;
  int list_max = n_idx;
  if (per_seq) {
    if (!union_done)
      DV_LAUNCH("union", hs, launch_union(idx, B, n_idx, m->n, o.U, o.cnt, masked ? o.mask : nullptr, hs));
    list = o.U;
    list_count = o.cnt;
    list_max = o.umax;
  }
  MrowsArgs r{};
  r.d = m->d; r.Kpad = o.Kpad; r.Ks = o.Ks; r.S = o.S; r.X = o.X16; r.mode = kRowsList;
  r.W0 = m->W1T; r.list = list; r.list_count = list_count; r.list_max = list_max; r.list_range = m->n;
  r.P = o.P; r.nrows_pad = o.nrows_pad; r.B = B;
  DV_LAUNCH("fc1", hs, launch_mrows(NB, r, hs));
  Fc1FinishArgs f{};
  f.P = o.P; f.S = o.S; f.nrows_pad = o.nrows_pad; f.list = list; f.list_count = list_count;
  f.list_max = list_max; f.list_range = m->n; f.b1 = m->b1; f.mask = (per_seq && masked) ? o.mask : nullptr; f.B = B;
  f.act = m->act;
  f.C = o.C; f.ldc = o.ldc;
  DV_LAUNCH("fc1_finish", hs, launch_fc1_finish(NB, f, hs));
  McolsArgs c{};
  c.d = m->d; c.M = m->W2T; c.list = list; c.list_count = list_count; c.list_max = list_max; c.dh = 0;
  c.list_range = m->n;
  c.C = o.C; c.ldc = o.ldc; c.S = o.S2; c.B = B; c.P = o.P2;
  DV_LAUNCH("fc2", hs, launch_mcols(NB, c, hs));
  ColsFinishArgs e{};
  e.P = o.P2; e.S = o.S2; e.B = B; e.d = m->d; e.bias = m->b2; e.resid = resid; e.out = out;
  DV_LAUNCH("fc2_finish", hs, launch_cols_finish(e, hs));
  return DV_OK;
}

dv_status batch_mlp(const dv_mlp* m, const float* x, int B, const int32_t* idx, int n_idx, int per_seq,
                    int batch_mode, float* out, void* ws, size_t ws_bytes, uint32_t flags, hipStream_t hs) {
  Workspace w(ws);
  BMlp o;
  if (bmlp_layout(m->d, m->n, B, n_idx, per_seq != 0, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  if (flags & DV_VALIDATE) {
    const dv_status st = validate_sets_sync(idx, per_seq ? B : 1, n_idx, m->n, o.cnt, hs);
    if (st != DV_OK) return st;
  }
  const bool masked = batch_mode == DV_MLP_MASKED;
  if (per_seq) {
    DV_LAUNCH("xcast_union", hs, launch_cast_union(x, B, batch_nb(B), m->d, o.Kpad, nullptr, nullptr, 0.f, o.X16, idx,
                                                   n_idx, m->n, o.U, o.cnt, masked ? o.mask : nullptr, hs));
    return bmlp_run(m, o, B, idx, n_idx, true, masked, nullptr, out, hs, true);
  }
  DV_LAUNCH("xcast", hs, launch_ln_cast(x, B, batch_nb(B), m->d, o.Kpad, nullptr, nullptr, 0.f, o.X16, hs));
  return bmlp_run(m, o, B, idx, n_idx, false, masked, nullptr, out, hs);
}

// ---------------------------------------------------------------- attention
struct BAttn {
  _Float16* X16; int32_t* Uh; int32_t* hcnt; float* P; float* q; float* part;
  _Float16* C;
  float* P2;
  int Kpad, S, Ks, nrows_pad, ldc, S2;
};

static size_t battn_layout(const dv_attn* a, int B, int n_heads, Workspace& w, BAttn* o) {
  const int NB = batch_nb(B);
  o->Kpad = round_up(a->d, 32);
  mrows_split(o->Kpad, NB, &o->S, &o->Ks);
  o->nrows_pad = round_up(3 * a->H * a->dh, 16);
  o->ldc = round_up(a->H * a->dh, 64);
  o->S2 = mcols_split(a->d, a->H * a->dh);
  o->X16 = w.take<_Float16>((size_t)NB * o->Kpad * 2);
  o->Uh = w.take<int32_t>((size_t)a->H * 4);
  o->hcnt = w.take<int32_t>(4);
  o->P = w.take<float>((size_t)o->S * o->nrows_pad * NB * 4);
  o->q = w.take<float>((size_t)B * std::max(n_heads, 1) * a->dh * 4);
  o->part = w.take<float>((size_t)B * std::max(n_heads, 1) * kAttnMaxSplit * (a->dh + 2) * 4);
  o->C = w.take<_Float16>((size_t)NB * o->ldc * 2);
  o->P2 = w.take<float>((size_t)o->S2 * B * a->d * 4);
  return w.off;
}

size_t batch_attn_ws(const dv_attn* a, int B, int n_heads) {
  Workspace w(nullptr);
  BAttn o;
  return battn_layout(a, B, n_heads, w, &o);
}

// Attention of every sequence on x16 (normalised fp16 [NB][Kpad]) for head sets
// heads[B][n_heads]; out = resid + bo + sum_{h in S_A^b} H_h W^O_h.
// union_done: the head union was built by the launch that cast x.
static dv_status battn_run(const dv_attn* a, const dv_kv* kv, const BAttn& o, int B, const int32_t* heads,
                           int n_heads, float scale, const float* resid, float* out, hipStream_t hs,
                           bool union_done = false) {
  const int NB = batch_nb(B);
  if (n_heads == 0) {
    ColsFinishArgs e{};
    e.P = nullptr; e.S = 0; e.B = B; e.d = a->d; e.bias = a->bo; e.resid = resid; e.out = out;
    DV_LAUNCH("oproj_finish", hs, launch_cols_finish(e, hs));
    return DV_OK;
  }
  if (!union_done) DV_LAUNCH("union_heads", hs, launch_union(heads, B, n_heads, a->H, o.Uh, o.hcnt, nullptr, hs));
  MrowsArgs r{};
  r.d = a->d; r.Kpad = o.Kpad; r.Ks = o.Ks; r.S = o.S; r.X = o.X16; r.mode = kRowsHeads;
  r.W0 = a->Wq; r.W1 = a->Wk; r.W2 = a->Wv; r.list = o.Uh; r.list_count = o.hcnt; r.list_max = a->H;
  r.list_range = a->H;
  r.dh = a->dh; r.P = o.P; r.nrows_pad = o.nrows_pad; r.B = B;
  DV_LAUNCH("qkv", hs, launch_mrows(NB, r, hs));
  QkvFinishArgs qf{};
  qf.P = o.P; qf.S = o.S; qf.nrows_pad = o.nrows_pad; qf.heads = heads; qf.n_heads = n_heads; qf.H = a->H;
  qf.dh = a->dh; qf.cap = kv->cap; qf.B = B; qf.hlist = o.Uh; qf.hcount = o.hcnt;
  qf.bq = a->bq; qf.bk = a->bk; qf.bv = a->bv; qf.q = o.q; qf.K = kv->K; qf.V = kv->V;
  int maxpos = 0;
  for (int b = 0; b < B; ++b) {
    qf.posb[b] = kv->pos[b];
    maxpos = std::max(maxpos, kv->pos[b]);
  }
  AttnArgs at{};
  at.H = a->H; at.dh = a->dh; at.cap = kv->cap; at.n_heads = n_heads;
  for (int b = 0; b < B; ++b) at.posb[b] = kv->pos[b];
  at.chunk = attn_chunk(B * n_heads, maxpos + 1, a->dh, kv->ktype);
  at.n_split = (maxpos + 1 + at.chunk - 1) / at.chunk;
  at.q = o.q; at.heads = heads; at.K = kv->K; at.V = kv->V; at.scale = scale; at.part = o.part;
  // One chunk per head (many sequences): the attention writes the coefficients itself,
  // into a matrix the QKV finisher clears; otherwise a launch combines the chunks.
  const bool direct = at.n_split == 1;
  if (direct && B > 1) {
    // Balance the CUs. At up to 4 (sequence, head) workgroups per CU (batch 32 with 32
    // heads each: all resident from the start) workgroup w runs on XCD w mod 8 and the
    // CUs of an XCD take its workgroups in turn, so a CU's share is the slots z0 + P j
    // (P = CUs / heads per sequence: the workgroups of one round of one per CU) and its
    // time the sum of their sequences' lengths, which differ up to 4x. Slots get the
    // sequences by decreasing length, every other row of P slots reversed, so a CU's
    // rows alternate long and short; with more workgroups than fit, dispatch then starts
    // the long ones first. Batch 32, lengths U[512, 2048]: 115 -> 107 us (104 us with
    // equal lengths).
    int idx[kMaxBatch];
    for (int b = 0; b < B; ++b) idx[b] = b;
    std::stable_sort(idx, idx + B, [&](int x, int y) { return kv->pos[x] > kv->pos[y]; });
    const int P = std::max(1, device_cu_count() / std::max(n_heads, 1));
    for (int z = 0; z < B; ++z) {
      const int row = z / P, s0 = z % P;
      const bool rev = (row & 1) && row * P + P <= B;
      at.seq_of[z] = idx[rev ? row * P + (P - 1 - s0) : z];
    }
    at.reorder = 1;
  }
  if (direct) {
    qf.zero = o.C; qf.zero_n = NB * o.ldc;
    at.C = o.C; at.ldc = o.ldc; at.cnb = NB; at.ulist = o.Uh; at.ucount = o.hcnt;
  }
  DV_LAUNCH("qkv_finish", hs, launch_qkv_finish(NB, kv->ktype, qf, hs));
  DV_LAUNCH("attn", hs, launch_attn(kv->ktype, at, B, hs));
  if (!direct) {
    AttnFinishArgs af{};
    af.part = o.part; af.n_split = at.n_split; af.n_heads = n_heads; af.dh = a->dh; af.B = B; af.heads = heads;
    af.list = o.Uh; af.hcount = o.hcnt; af.C = o.C; af.ldc = o.ldc;
    DV_LAUNCH("attn_finish", hs, launch_attn_finish(NB, af, hs));
  }
  McolsArgs c{};
  c.d = a->d; c.M = a->WoT; c.list = o.Uh; c.list_count = o.hcnt; c.list_max = a->H; c.dh = a->dh;
  c.list_range = a->H;
  c.C = o.C; c.ldc = o.ldc; c.S = o.S2; c.B = B; c.P = o.P2;
  DV_LAUNCH("oproj", hs, launch_mcols(NB, c, hs));
  ColsFinishArgs e{};
  e.P = o.P2; e.S = o.S2; e.B = B; e.d = a->d; e.bias = a->bo; e.resid = resid; e.out = out;
  DV_LAUNCH("oproj_finish", hs, launch_cols_finish(e, hs));
  return DV_OK;
}

dv_status batch_attn(const dv_attn* a, const float* x, int B, const dv_kv* kv, const int32_t* heads, int n_heads,
                     float scale, float* out, void* ws, size_t ws_bytes, uint32_t flags, hipStream_t hs) {
  Workspace w(ws);
  BAttn o;
  if (battn_layout(a, B, n_heads, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  if (flags & DV_VALIDATE) {
    const dv_status st = validate_sets_sync(heads, B, n_heads, a->H, o.hcnt, hs);
    if (st != DV_OK) return st;
  }
  if (n_heads > 0)
    DV_LAUNCH("xcast_union_heads", hs, launch_cast_union(x, B, batch_nb(B), a->d, o.Kpad, nullptr, nullptr, 0.f, o.X16,
                                                         heads, n_heads, a->H, o.Uh, o.hcnt, nullptr, hs));
  return battn_run(a, kv, o, B, heads, n_heads, scale, nullptr, out, hs, true);
}

// ---------------------------------------------------------------- layer
struct BBlock {
  BAttn at;        // X16 doubles as LN1(y) and, later, LN2(y~)
  BMlp ml;         // shares nothing with `at` (both live for the whole call)
  _Float16* Hh16; _Float16* Hm16; float* Pp; float* s_h; float* s_m; int32_t* heads; int32_t* idx; float* yt;
  int ldr0, ldr1, Sp, Ksp, rows_p;
};

static size_t bblock_layout(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa, const dv_predictor* pm,
                            int B, int kh, int km, Workspace& w, BBlock* o) {
  const int NB = batch_nb(B);
  battn_layout(a, B, kh, w, &o->at);
  bmlp_layout(m->d, m->n, B, km, true, w, &o->ml);
  o->ldr0 = round_up(pa->r, 32);
  o->ldr1 = round_up(pm->r, 32);
  const int Kpad = round_up(a->d, 32);
  mrows_split(Kpad, NB, &o->Sp, &o->Ksp);
  o->rows_p = round_up(pa->r + pm->r, 16);
  o->Pp = w.take<float>((size_t)o->Sp * o->rows_p * NB * 4);
  o->Hh16 = w.take<_Float16>((size_t)NB * o->ldr0 * 2);
  o->Hm16 = w.take<_Float16>((size_t)NB * o->ldr1 * 2);
  o->s_h = w.take<float>((size_t)B * a->H * 4);
  o->s_m = w.take<float>((size_t)B * m->n * 4);
  o->heads = w.take<int32_t>((size_t)B * kh * 4);
  o->idx = w.take<int32_t>((size_t)B * km * 4);
  o->yt = w.take<float>((size_t)B * a->d * 4);
  return w.off;
}

size_t batch_block_ws(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa, const dv_predictor* pm, int B,
                      int kh, int km) {
  Workspace w(nullptr);
  BBlock o;
  return bblock_layout(a, m, pa, pm, B, kh, km, w, &o);
}

// The largest predictor rank the batched scores stage takes in one K split.
int batch_max_rank(int B) {
  int S = 0, Ks = 0;
  const int unit = 32 * 8;
  for (int r = unit;; r += unit) {
    mrows_split(r, batch_nb(B), &S, &Ks);
    if (S > 1) return r - unit;
  }
}

// Predictor hidden layers (one or two predictors on the same x16) and their scores.
static dv_status bpredict(const BBlock& o, const _Float16* x16, int d, int B, const dv_predictor* p0, _Float16* h0,
                          int ld0, float* s0, const dv_predictor* p1, _Float16* h1, int ld1, float* s1,
                          hipStream_t hs) {
  const int NB = batch_nb(B);
  MrowsArgs r{};
  r.d = d; r.Kpad = round_up(d, 32); r.Ks = o.Ksp; r.S = o.Sp; r.X = x16; r.mode = kRowsIdentity;
  r.W0 = p0->AT; r.n0 = p0->r; r.W1 = p1 ? p1->AT : nullptr; r.nrows = p0->r + (p1 ? p1->r : 0);
  r.P = o.Pp; r.nrows_pad = o.rows_p; r.B = B;
  DV_LAUNCH("pred_hidden", hs, launch_mrows(NB, r, hs));
  DV_LAUNCH("pred_hidden_cast", hs, launch_sum_cast(NB, o.Pp, o.Sp, o.rows_p, 0, p0->r, B, h0, ld0, hs));
  if (p1) DV_LAUNCH("pred_hidden_cast", hs, launch_sum_cast(NB, o.Pp, o.Sp, o.rows_p, p0->r, p1->r, B, h1, ld1, hs));
  const dv_predictor* ps[2] = {p0, p1};
  const _Float16* hx[2] = {h0, h1};
  const int lds[2] = {ld0, ld1};
  float* sc[2] = {s0, s1};
  for (int i = 0; i < 2; ++i) {
    if (ps[i] == nullptr) continue;
    MrowsArgs q{};
    q.d = ps[i]->r; q.Kpad = lds[i];
    mrows_split(q.Kpad, NB, &q.S, &q.Ks);
    if (q.S != 1) return DV_ERR_UNSUPPORTED;
    q.X = hx[i]; q.mode = kRowsIdentity; q.W0 = ps[i]->BT; q.n0 = ps[i]->n_out; q.nrows = ps[i]->n_out;
    q.out0 = sc[i]; q.ld0 = ps[i]->n_out; q.B = B;
    DV_LAUNCH("pred_scores", hs, launch_mrows(NB, q, hs));
  }
  return DV_OK;
}

dv_status batch_block(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa, const dv_predictor* pm,
                      const dv_ln* ln, const dv_kv* kv, const float* x_in, float* x_out, int B, int kh, int km,
                      int mode, int batch_mode, float scale, int32_t* heads_out, int32_t* idx_out, void* ws,
                      size_t ws_bytes, hipStream_t hs) {
  Workspace w(ws);
  BBlock o;
  if (bblock_layout(a, m, pa, pm, B, kh, km, w, &o) > ws_bytes) return DV_ERR_WORKSPACE;
  const int NB = batch_nb(B);
  const bool ahead = mode == DV_LOOKAHEAD;
  const float* g1 = ln ? ln->g1 : nullptr;
  const float* be1 = ln ? ln->be1 : nullptr;
  const float* g2 = ln ? ln->g2 : nullptr;
  const float* be2 = ln ? ln->be2 : nullptr;
  const float eps = ln ? ln->eps : 0.f;
  dv_status st;
  // 1. LN1(y) as fp16; predictors (both in look-ahead mode) and their top-k sets.
  DV_LAUNCH("ln1", hs, launch_ln_cast(x_in, B, NB, a->d, o.at.Kpad, g1, be1, eps, o.at.X16, hs));
  st = bpredict(o, o.at.X16, a->d, B, pa, o.Hh16, o.ldr0, o.s_h, ahead ? pm : nullptr, o.Hm16, o.ldr1, o.s_m, hs);
  if (st != DV_OK) return st;
  DV_LAUNCH("select_heads", hs,
            launch_select(o.s_h, B, a->H, DV_SELECT_TOPK, kh, 0.f, o.heads, kh, nullptr, heads_out, hs));
  if (ahead)
    DV_LAUNCH("select_mlp", hs,
              launch_select(o.s_m, B, m->n, DV_SELECT_TOPK, km, 0.f, o.idx, km, nullptr, idx_out, hs));
  // 2. y~ = y + MHA_{S_A}(LN1(y)).
  st = battn_run(a, kv, o.at, B, o.heads, kh, scale, x_in, o.yt, hs);
  if (st != DV_OK) return st;
  // 3. LN2(y~) as fp16 (into the MLP's x-hat buffer), with the union of the neuron sets
  //    in the same launch in look-ahead mode; sequential mode predicts S_M here.
  const bool masked = batch_mode == DV_MLP_MASKED;
  if (ahead)
    DV_LAUNCH("ln2_union", hs, launch_cast_union(o.yt, B, NB, m->d, o.ml.Kpad, g2, be2, eps, o.ml.X16, o.idx, km,
                                                 m->n, o.ml.U, o.ml.cnt, masked ? o.ml.mask : nullptr, hs));
  else
    DV_LAUNCH("ln2", hs, launch_ln_cast(o.yt, B, NB, m->d, o.ml.Kpad, g2, be2, eps, o.ml.X16, hs));
  if (!ahead) {
    st = bpredict(o, o.ml.X16, m->d, B, pm, o.Hm16, o.ldr1, o.s_m, nullptr, nullptr, 0, nullptr, hs);
    if (st != DV_OK) return st;
    DV_LAUNCH("select_mlp", hs,
              launch_select(o.s_m, B, m->n, DV_SELECT_TOPK, km, 0.f, o.idx, km, nullptr, idx_out, hs));
  }
  // 4. y^ = y~ + MLP_{S_M}(LN2(y~)) on the union of the sets.
  return bmlp_run(m, o.ml, B, o.idx, km, true, masked, o.yt, x_out, hs, ahead);
}

}  // namespace dv
