// Sparsity predictors (Sections 4.1-4.2): s = (x A) B, then top-k or threshold
// selection. A = AT^T is d x r and B = BT^T is r x n; both factors are stored with
// their output index as the row so every GEMV streams whole contiguous rows.
#include "dv_internal.hpp"
#include "dv_rowdot.hpp"
#include "dv_select.hpp"

namespace dv {

// ----------------------------------------------------------- hidden layer
// h[b][j] = x-hat[b] . AT[j] for the rows of up to two predictors; one workgroup per
// CU takes a contiguous range of rows whose loads its wavefronts split evenly.
template <typename T, int NW, int U, int KX, bool LN>
__global__ void __launch_bounds__(NW * 64) k_pred_hidden(PredHidArgs a) {
  extern __shared__ float smem[];
  float* xs = smem;
  float* red = smem + a.d;
  float* part = red + NW;
  const int b = blockIdx.y;
  auto row_ptr = [&](int row) {
    return row < a.r0 ? static_cast<const T*>(a.AT0) + (size_t)row * a.d
                      : static_cast<const T*>(a.AT1) + (size_t)(row - a.r0) * a.d;
  };
  auto epi = [&](int row, float v) {
    if (row < a.r0)
      a.hid0[(size_t)b * a.r0 + row] = v;
    else
      a.hid1[(size_t)b * a.r1 + row - a.r0] = v;
  };
  rowdot_flat<T, NW, U, KX, LN>(row_ptr, epi, a.r0 + a.r1, a.d, a.x + (size_t)b * a.d, a.g, a.be, a.eps, xs, red, part,
                        a.xhat_out ? a.xhat_out + (size_t)b * a.d : nullptr, blockIdx.x, gridDim.x);
}

template <typename T, int KX>
static hipError_t launch_pred_hidden_t(const PredHidArgs& a, hipStream_t st) {
  // two batches of 2 loads in flight per wavefront: measured faster than all of a
  // wavefront's loads at once (12 at the OPT-175B shape) or batches of 1, 3, 4 or 6,
  // as deeper queues let the XCDs that win the fabric arbitration run ahead
  constexpr int NW = 16, U = 2;
  const int nrows = a.r0 + a.r1;
  const dim3 grid(max(1, min(nrows, device_cu_count())), a.B);
  const size_t lds = (size_t)(a.d + NW + rowdot_flat_part(nrows, grid.x, NW)) * sizeof(float);
  const void* kern = a.g != nullptr ? reinterpret_cast<const void*>(k_pred_hidden<T, NW, U, KX, true>)
                                    : reinterpret_cast<const void*>(k_pred_hidden<T, NW, U, KX, false>);
  const hipError_t e = ensure_dyn_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (a.g != nullptr)
    launch_k((k_pred_hidden<T, NW, U, KX, true>), grid, dim3(NW * 64), lds, st, a);
  else
    launch_k((k_pred_hidden<T, NW, U, KX, false>), grid, dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_pred_hidden_k(const PredHidArgs& a, hipStream_t st) {
  switch (rowdot_kx(a.d, 16)) {
    case 1: return launch_pred_hidden_t<T, 1>(a, st);
    case 2: return launch_pred_hidden_t<T, 2>(a, st);
    case 3: return launch_pred_hidden_t<T, 3>(a, st);
    default: return launch_pred_hidden_t<T, 4>(a, st);
  }
}

hipError_t launch_pred_hidden(int wtype, const PredHidArgs& a, hipStream_t st) {
  return wtype == DV_F16 ? launch_pred_hidden_k<_Float16>(a, st) : launch_pred_hidden_k<float>(a, st);
}

// ----------------------------------------------------------------- scores
// G lanes per row (a row is r elements, short); RU rows per lane group in flight.
// With a.sel_k0 > 0 workgroup 0 takes all rows of the first predictor (the head
// predictor, n0 <= NT) and selects its top-k set right away, so that the next kernel
// finds the head set ready; the other workgroups take the remaining rows.
// Head workgroup of a hosted selection: the n0 rows of the first predictor, RB rows
// per wavefront per round with every load of a round in flight before the input is
// staged (one round trip at H <= RB * NW; the workgroup runs beside a kernel that
// saturates HBM, where each round trip is slow), then the top-k set.
template <typename T, int NW, int RB>
__device__ __forceinline__ void head_scores_select(const PredScoreArgs& a, float* xs0, float* hsc) {
  constexpr int NT = NW * 64;
  constexpr int E = Chunk<T>::E;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = a.r0 / E;                      // r0 <= 1536 for a hosted selection
  const char* base = static_cast<const char*>(a.BT0);
  const size_t rowb = (size_t)a.r0 * sizeof(T);
  bool staged = false;
  for (int r0 = wave; r0 - wave < a.n0; r0 += NW * RB) {
    u32x4 w[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = min(r0 + rb * NW, a.n0 - 1);
#pragma unroll
      for (int h = 0; h < 2; ++h) w[rb][h] = ld_stream(base + row * rowb + (size_t)min(h * 64 + lane, nch - 1) * 16);
    }
    if (!staged) {
      stage_x<T, NT>(a.hid0, a.r0, xs0);
      staged = true;
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = r0 + rb * NW;
      float acc = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = h * 64 + lane;
        if (c < nch) acc = dot_chunk<T>(w[rb][h], xs0, a.r0, c, acc);
      }
      acc = wave_sum(acc);
      if (lane == 0 && row < a.n0) {
        hsc[row] = acc;
        a.s0[row] = acc;
      }
    }
  }
  if (!staged) stage_x<T, NT>(a.hid0, a.r0, xs0);   // (no rows: keep barriers)
  uint32_t* keys = reinterpret_cast<uint32_t*>(hsc + a.n0);
  int* tmp = reinterpret_cast<int*>(keys + a.n0);
  int32_t* set = tmp + a.n0;
  __syncthreads();
  wg_topk_small<NT>(hsc, a.n0, a.sel_k0, keys, tmp, set);
  for (int i = threadIdx.x; i < a.sel_k0; i += NT) {
    a.sel_set0[i] = set[i];
    if (a.sel_set0_out) a.sel_set0_out[i] = set[i];
  }
}

// The grid is sized to stay resident (two workgroups per CU); workgroup wg of G takes
// a contiguous share of the rows (the second half of the grid smaller shares, below)
// and its wavefronts split that share evenly.
// A wavefront works in groups of RU rows per lane group (GPW = 64 / G groups of G
// lanes); every load of a group (NR rounds of G chunks per row, row and chunk
// clamped, surplus masked where summed) is issued before the group is used, and
// with one round of chunks per row two groups are in flight. With EARLY (ranks up to 4 * NT) the
// first group's loads go out before the hidden vectors are staged: their reads are
// issued first, as straight-line code, so that the staging waits for them alone and
// the weight stream starts at once instead of after their round trip.
template <typename T, int NW, int G, int RU, int NR, bool EARLY>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2 * NW / 4))) k_pred_scores(PredScoreArgs a) {
  extern __shared__ float smem[];
  constexpr int NT = NW * 64;
  constexpr int E = Chunk<T>::E;
  const int b = blockIdx.y;
  const int r0a = (a.r0 + 3) & ~3;
  float* xs0 = smem;
  float* xs1 = smem + r0a;
  const bool hosted = a.sel_k0 > 0;
  if (hosted && blockIdx.x == 0) {
    head_scores_select<T, NW, 6>(a, xs0, xs1 + ((a.r1 + 3) & ~3));
    return;
  }
  const bool two = a.n1 > 0;
  StageX<T, NT, 1> hx0, hx1;
  if constexpr (EARLY) {
    hx0.load(a.hid0 + (size_t)b * a.r0, a.r0, nullptr, nullptr);
    // (one predictor: a read that is unused and not the first one's, so that the
    // compiler does not fold the two into a wait and a branch)
    hx1.load(two ? a.hid1 + (size_t)b * a.r1 : a.hid0 + (size_t)b * a.r0, two ? a.r1 : 4, nullptr, nullptr);
  } else {
    stage_x<T, NT>(a.hid0 + (size_t)b * a.r0, a.r0, xs0);
    if (two) stage_x<T, NT>(a.hid1 + (size_t)b * a.r1, a.r1, xs1);
  }
  const int nrows = a.n0 + a.n1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int grp = lane / G, gl = lane % G;
  constexpr int GPW = 64 / G;          // row groups per wavefront
  constexpr int RPG = GPW * RU;        // rows per wavefront group
  const int Gw = (int)gridDim.x - (hosted ? 1 : 0), wg = (int)blockIdx.x - (hosted ? 1 : 0);
  const int rb = hosted ? a.n0 : 0, R = nrows - rb;
  // Workgroups of the second half start their stream later (they are dispatched
  // second, onto CUs whose first workgroup already has its loads in flight, and their
  // hidden-vector reads queue behind them), so they take 15 % fewer rows than those of
  // the first half (per-workgroup clocks at the OPT-175B predictors: last end 20.0 ->
  // 18.9 us; 0.4 us off the launch).
  auto cum = [&](int i) -> long {
    const int h = Gw / 2;
    return i <= h ? (long)i * 115 : (long)h * 115 + (long)(i - h) * 85;
  };
  const int w0 = rb + (int)((long)R * cum(wg) / cum(Gw)), w1 = rb + (int)((long)R * cum(wg + 1) / cum(Gw));
  const int v0 = w0 + (w1 - w0) * wave / NW, v1 = w0 + (w1 - w0) * (wave + 1) / NW;   // this wavefront's rows
  const int ng = (v1 - v0 + RPG - 1) / RPG;
  if (!EARLY && ng == 0) return;
  const int nch0 = a.r0 / E, nch1 = a.r1 / E;
  const int cmax = max(nch0, a.n1 > 0 ? nch1 : 0);

  auto row_of = [&](int k, int u) { return v0 + k * RPG + u * GPW + grp; };
  auto load = [&](u32x4 (&w)[RU][NR], int k, int c0) {
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int row = max(min(row_of(k, u), v1 - 1), 0);   // (a wavefront without rows reads row 0)
      const bool sec = row >= a.n0;
      const char* rp = sec ? reinterpret_cast<const char*>(static_cast<const T*>(a.BT1) + (size_t)(row - a.n0) * a.r1)
                           : reinterpret_cast<const char*>(static_cast<const T*>(a.BT0) + (size_t)row * a.r0);
      const int nch = sec ? nch1 : nch0;
#pragma unroll
      for (int h = 0; h < NR; ++h) w[u][h] = ld_stream(rp + (size_t)min(c0 + h * G + gl, nch - 1) * 16);
    }
  };
  auto consume = [&](const u32x4 (&w)[RU][NR], int k, int c0) {
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int row = row_of(k, u);
      const bool sec = row >= a.n0;
      const int nch = sec ? nch1 : nch0;
      float acc = 0.f;
#pragma unroll
      for (int h = 0; h < NR; ++h) {
        const int c = c0 + h * G + gl;
        if (c < nch) acc = sec ? dot_chunk<T>(w[u][h], xs1, a.r1, c, acc) : dot_chunk<T>(w[u][h], xs0, a.r0, c, acc);
      }
#pragma unroll
      for (int o = G / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kWave);
      if (gl == 0 && row < v1) {
        float* out = sec ? a.s1 + (size_t)b * a.n1 + row - a.n0 : a.s0 + (size_t)b * a.n0 + row;
        *out = c0 == 0 ? acc : *out + acc;   // rows longer than NR * G chunks: one round per c0
      }
    }
  };
  u32x4 w[RU][NR];
  if constexpr (EARLY) {
    load(w, 0, 0);   // the first group, before the staging waits
    hx0.finish(a.r0, false, 0.f, xs0, nullptr);
    if (two) hx1.finish(a.r1, false, 0.f, xs1, nullptr);
    if (ng == 0) return;
  }
  if (cmax <= NR * G) {
    // one round of chunks (the usual case): groups alternate between two register
    // sets, the next group's loads issued before the current group is used
    u32x4 w2[RU][NR];
    if (!EARLY) load(w, 0, 0);
    for (int k = 0; k < ng; k += 2) {
      if (k + 1 < ng) load(w2, k + 1, 0);
      consume(w, k, 0);
      if (k + 1 >= ng) break;
      if (k + 2 < ng) load(w, k + 2, 0);
      consume(w2, k + 1, 0);
    }
    return;
  }
  for (int c0 = 0; c0 < cmax; c0 += NR * G) {
    for (int k = 0; k < ng; ++k) {
      if (!EARLY || c0 > 0 || k > 0) load(w, k, c0);
      consume(w, k, c0);
    }
  }
}

// (ranks of two predictors staged together pass 64 KB: up to 2 x 16000 floats)
template <typename T, int NW, int G, int RU, int NR, bool EARLY>
static hipError_t launch_scores_k(const PredScoreArgs& a, dim3 grid, size_t lds, hipStream_t st) {
  const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(k_pred_scores<T, NW, G, RU, NR, EARLY>), lds);
  if (e != hipSuccess) return e;
  launch_k((k_pred_scores<T, NW, G, RU, NR, EARLY>), grid, dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_scores_t(const PredScoreArgs& a, hipStream_t st) {
  constexpr int NW = 8;
  constexpr int E = Chunk<T>::E;
  const int nch = max(a.r0, a.r1) / E;
  const int nrows = a.n0 + a.n1;
  const int hosted = a.sel_k0 > 0 ? 1 : 0;
  const size_t lds = (size_t)(((a.r0 + 3) & ~3) + ((a.r1 + 3) & ~3) + 4 * a.n0 * hosted + 4) * sizeof(float);
  // two workgroups per CU (the head-selection workgroup included): all resident at once
  const int blocks = max(1, min(2 * device_cu_count() - hosted, nrows));
  const dim3 grid(blocks + hosted, a.B);
  // hidden vectors staged behind the first loads when one float4 per thread holds them
  const bool early = max(a.r0, a.r1) <= 4 * NW * 64;
  if (nch > 32) {
    // 64 lanes per row, all chunks of a row up to 128 (r <= 1024 fp16) in one round;
    // groups of 2 rows, two in flight (measured fastest; groups of 1, 4 or 13 rows were slower)
    return early ? launch_scores_k<T, NW, 64, 2, 2, true>(a, grid, lds, st)
                 : launch_scores_k<T, NW, 64, 2, 2, false>(a, grid, lds, st);
  } else if (nch > 16) {
    return early ? launch_scores_k<T, NW, 32, 8, 1, true>(a, grid, lds, st)
                 : launch_scores_k<T, NW, 32, 8, 1, false>(a, grid, lds, st);
  }
  return early ? launch_scores_k<T, NW, 16, 8, 1, true>(a, grid, lds, st)
               : launch_scores_k<T, NW, 16, 8, 1, false>(a, grid, lds, st);
}

hipError_t launch_pred_scores(int wtype, const PredScoreArgs& a, hipStream_t st) {
  return wtype == DV_F16 ? launch_scores_t<_Float16>(a, st) : launch_scores_t<float>(a, st);
}

// ---------------------------------------------------------------- select
__global__ void __launch_bounds__(1024) k_select(const float* s, int n, int mode, int k, float thresh,
                                                 int32_t* idx, int cap, int32_t* count, int32_t* idx2) {
  __shared__ uint32_t hist[kSelBins];
  __shared__ int sm[kSelSm(1024)];
  const int b = blockIdx.x;
  if (n <= 1024)
    wg_select_small<1024>(s + (size_t)b * n, n, mode, k, thresh, idx + (size_t)b * cap, cap,
                          count ? count + b : nullptr, idx2 ? idx2 + (size_t)b * cap : nullptr, hist, sm);
  else if (n <= 1024 * 48)
    wg_select_reg<1024, 48>(s + (size_t)b * n, n, mode, k, thresh, idx + (size_t)b * cap, cap,
                            count ? count + b : nullptr, idx2 ? idx2 + (size_t)b * cap : nullptr, hist, sm);
  else
    wg_select<1024>(s + (size_t)b * n, n, mode, k, thresh, idx + (size_t)b * cap, cap,
                    count ? count + b : nullptr, idx2 ? idx2 + (size_t)b * cap : nullptr, hist, sm);
}

hipError_t launch_select(const float* scores, int B, int n, int mode, int k, float thresh,
                         int32_t* idx, int cap, int32_t* count, int32_t* idx2, hipStream_t st) {
  launch_k(k_select, dim3(B), dim3(1024), 0, st, scores, n, mode, k, thresh, idx, cap, count, idx2);
  return hipGetLastError();
}

// One workgroup checks every set: strictly ascending and within [0, range).
// A debugging aid (DV_VALIDATE), not on the timed path.
__global__ void __launch_bounds__(1024) k_validate_sets(const int32_t* set, int B, int n, int range,
                                                        int32_t* bad) {
  __shared__ int any_bad;
  if (threadIdx.x == 0) any_bad = 0;
  __syncthreads();
  int ok = 1;
  const long total = (long)B * n;
  for (long g = threadIdx.x; g < total; g += 1024) {
    const int i = (int)(g % n);
    const int v = set[g];
    ok &= (v >= 0) & (v < range);
    if (i > 0) ok &= set[g - 1] < v;
  }
  if (!ok) atomicOr(&any_bad, 1);
  __syncthreads();
  if (threadIdx.x == 0) *bad = any_bad;
}

hipError_t launch_validate_sets(const int32_t* set, int B, int n, int range, int32_t* bad, hipStream_t st) {
  launch_k(k_validate_sets, dim3(1), dim3(1024), 0, st, set, B, n, range, bad);
  return hipGetLastError();
}

}  // namespace dv

// ------------------------------------------------------------------ C ABI
using namespace dv;

static dv_status check_predictor(const dv_predictor* p) {
  if (p == nullptr || p->AT == nullptr || p->BT == nullptr) return DV_ERR_NULL;
  if (p->wtype != DV_F16 && p->wtype != DV_F32) return DV_ERR_DTYPE;
  if (p->d <= 0 || p->r <= 0 || p->n_out <= 0) return DV_ERR_SHAPE;
  const int E = 16 / elem_bytes(p->wtype);
  if (p->d % E != 0 || p->r % E != 0) return DV_ERR_ALIGN;
  if (!aligned16(p->AT) || !aligned16(p->BT)) return DV_ERR_ALIGN;
  if (p->d > 16000 || p->r > 16000) return DV_ERR_UNSUPPORTED;   // LDS staging budget
  if (p->n_out > (1 << 26)) return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

static size_t predict_ws(const dv_predictor* p, int32_t B, float* scores_given, Workspace& w,
                         float** hid, float** scores) {
  *hid = w.take<float>((size_t)B * p->r * sizeof(float));
  float* s = w.take<float>(scores_given ? 0 : (size_t)B * p->n_out * sizeof(float));
  *scores = scores_given ? scores_given : s;
  return w.off;
}

extern "C" size_t dv_predict_workspace_bytes(const dv_predictor* p, int32_t B) {
  if (p == nullptr || B <= 0 || p->r <= 0 || p->n_out <= 0) return 0;
  Workspace w(nullptr);
  float *h, *s;
  return predict_ws(p, B, nullptr, w, &h, &s);
}

static dv_status predict_impl(const dv_predictor* p, const float* x, int32_t B, int32_t mode, int32_t k,
                              float thresh, int32_t* idx, int32_t cap_idx, int32_t* count, float* scores,
                              void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
  trace_reset();
  dv_status st = check_predictor(p);
  if (st != DV_OK) return st;
  if (x == nullptr || idx == nullptr) return DV_ERR_NULL;
  if (B <= 0 || B > 65535) return DV_ERR_SHAPE;
  if (!aligned16(x)) return DV_ERR_ALIGN;
  if (flags & ~(uint32_t)(DV_DETERMINISTIC | DV_VALIDATE)) return DV_ERR_ARG;
  if (mode == DV_SELECT_TOPK) {
    if (k < 0 || k > p->n_out || cap_idx < k) return DV_ERR_SHAPE;
  } else if (mode == DV_SELECT_THRESHOLD) {
    if (cap_idx < 0) return DV_ERR_SHAPE;
  } else {
    return DV_ERR_ARG;
  }
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return DV_ERR_WORKSPACE;
  Workspace w(ws);
  float *hid, *s;
  if (predict_ws(p, B, scores, w, &hid, &s) > ws_bytes) return DV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);

  PredHidArgs ha{};
  ha.d = p->d; ha.B = B; ha.x = x; ha.g = nullptr; ha.be = nullptr; ha.eps = 0.f;
  ha.AT0 = p->AT; ha.r0 = p->r; ha.hid0 = hid; ha.AT1 = nullptr; ha.r1 = 0; ha.hid1 = nullptr;
  DV_LAUNCH("pred_hidden", hs, launch_pred_hidden(p->wtype, ha, hs));
  PredScoreArgs sa{};
  sa.r0 = p->r; sa.n0 = p->n_out; sa.BT0 = p->BT; sa.hid0 = hid; sa.s0 = s;
  sa.r1 = 0; sa.n1 = 0; sa.B = B;
  DV_LAUNCH("pred_scores", hs, launch_pred_scores(p->wtype, sa, hs));
  DV_LAUNCH("select", hs, launch_select(s, B, p->n_out, mode, k, thresh, idx, cap_idx, count, nullptr, hs));
  return DV_OK;
}

extern "C" dv_status dv_predict_mlp(const dv_predictor* p, const float* x, int32_t B, int32_t mode,
                                    int32_t k, float thresh, int32_t* idx, int32_t cap_idx,
                                    int32_t* count, float* scores, void* ws, size_t ws_bytes,
                                    uint32_t flags, void* stream) {
  return predict_impl(p, x, B, mode, k, thresh, idx, cap_idx, count, scores, ws, ws_bytes, flags, stream);
}

extern "C" dv_status dv_predict_heads(const dv_predictor* p, const float* x, int32_t B, int32_t mode,
                                      int32_t k, float thresh, int32_t* idx, int32_t cap_idx,
                                      int32_t* count, float* scores, void* ws, size_t ws_bytes,
                                      uint32_t flags, void* stream) {
  return predict_impl(p, x, B, mode, k, thresh, idx, cap_idx, count, scores, ws, ws_bytes, flags, stream);
}
