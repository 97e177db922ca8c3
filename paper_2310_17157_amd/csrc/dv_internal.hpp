// Internal definitions shared by the HIP translation units of the Deja Vu decode
// library: device helpers (16-byte weight chunks, wavefront and workgroup
// reductions, layer-norm staging into LDS, order-preserving float keys), kernel
// argument structures and the host-side launchers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>

#include "dv.h"

namespace dv {

constexpr int kWave = 64;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// 4-bit weights (W4A16): a 16-byte chunk holds 32 elements, two per byte (low nibble
// first), element = scale * (code - 8), one fp16 scale per chunk kept in a separate
// array (scale of chunk c of a row: scales[row][c]).
struct q4_t {};

// Elements per 16-byte chunk for a storage type.
template <typename T> struct Chunk;
template <> struct Chunk<float> { static constexpr int E = 4; };
template <> struct Chunk<_Float16> { static constexpr int E = 8; };
template <> struct Chunk<q4_t> { static constexpr int E = 32; };
template <typename T> inline constexpr bool kIsQ4 = false;
template <> inline constexpr bool kIsQ4<q4_t> = true;

// Activation of the MLP (sigma of Eq. (1)).
enum { kActRelu = 0, kActGelu = 1 };
__device__ __forceinline__ float act_apply(float v, int act) {
  if (act == kActGelu) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v > 0.f ? v : 0.f;
}

// ---------------------------------------------------------------- loads
// Weights are streamed once per call: non-temporal 16-byte loads.
__device__ __forceinline__ u32x4 ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x4 ld_plain(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Unpack a 16-byte chunk into E floats.
template <typename T>
__device__ __forceinline__ void unpack(u32x4 w, float* v);
template <>
__device__ __forceinline__ void unpack<float>(u32x4 w, float* v) {
  f32x4 f = __builtin_bit_cast(f32x4, w);
  v[0] = f[0]; v[1] = f[1]; v[2] = f[2]; v[3] = f[3];
}
template <>
__device__ __forceinline__ void unpack<_Float16>(u32x4 w, float* v) {
  f16x8 h = __builtin_bit_cast(f16x8, w);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)h[i];
}

// A 4-bit chunk as 32 floats code - 8 (the caller applies the chunk's scale).
template <>
__device__ __forceinline__ void unpack<q4_t>(u32x4 w, float* v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int k = 0; k < 8; ++k) v[8 * i + k] = (float)((int)((w[i] >> (4 * k)) & 15u) - 8);
  }
}

// Store E floats as one chunk of storage type T (round to nearest even for fp16).
template <typename T>
__device__ __forceinline__ void store_elem(T* p, float v) { *p = (T)v; }

// ---------------------------------------------------- x-hat in LDS
// The input vector of a row-dot is staged in LDS as fp32. For fp16 rows a 16-byte
// chunk c holds elements 8c..8c+7; its fp32 operands live in two planes (elements
// 8c..8c+3 at plane 0, 8c+4..8c+7 at plane 1) so that lanes reading consecutive
// chunks read consecutive 16-byte words of each plane. For fp32 rows chunk c is
// elements 4c..4c+3 of a single plane.
template <typename T>
__device__ __forceinline__ int xs_index(int e, int d);
template <>
__device__ __forceinline__ int xs_index<float>(int e, int) { return e; }
template <>
__device__ __forceinline__ int xs_index<_Float16>(int e, int d) {
  return ((e >> 2) & 1) * (d >> 1) + ((e >> 3) << 2) + (e & 3);
}
// 4-bit rows: eight planes (elements 4p..4p+3 of every 32-element chunk in plane p).
template <>
__device__ __forceinline__ int xs_index<q4_t>(int e, int d) {
  return ((e >> 2) & 7) * (d >> 3) + ((e >> 5) << 2) + (e & 3);
}

template <typename T>
__device__ __forceinline__ float dot_chunk(u32x4 w, const float* xs, int d, int c, float acc);
template <>
__device__ __forceinline__ float dot_chunk<float>(u32x4 w, const float* xs, int, int c, float acc) {
  f32x4 wf = __builtin_bit_cast(f32x4, w);
  f32x4 x = *reinterpret_cast<const f32x4*>(xs + 4 * c);
  acc = fmaf(wf[0], x[0], acc);
  acc = fmaf(wf[1], x[1], acc);
  acc = fmaf(wf[2], x[2], acc);
  acc = fmaf(wf[3], x[3], acc);
  return acc;
}
template <>
__device__ __forceinline__ float dot_chunk<_Float16>(u32x4 w, const float* xs, int d, int c, float acc) {
  f16x8 h = __builtin_bit_cast(f16x8, w);
  f32x4 xa = *reinterpret_cast<const f32x4*>(xs + 4 * c);
  f32x4 xb = *reinterpret_cast<const f32x4*>(xs + (d >> 1) + 4 * c);
  acc = fmaf((float)h[0], xa[0], acc);
  acc = fmaf((float)h[1], xa[1], acc);
  acc = fmaf((float)h[2], xa[2], acc);
  acc = fmaf((float)h[3], xa[3], acc);
  acc = fmaf((float)h[4], xb[0], acc);
  acc = fmaf((float)h[5], xb[1], acc);
  acc = fmaf((float)h[6], xb[2], acc);
  acc = fmaf((float)h[7], xb[3], acc);
  return acc;
}

// Dot of a 4-bit chunk (scale sc) with its 32 staged inputs: sc * sum (code - 8) x.
__device__ __forceinline__ float dot_chunk_q4(u32x4 w, float sc, const float* xs, int d, int c, float acc) {
  float t = 0.f;
  const int plane = d >> 3;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x4 xa = *reinterpret_cast<const f32x4*>(xs + (2 * i) * plane + 4 * c);
    const f32x4 xb = *reinterpret_cast<const f32x4*>(xs + (2 * i + 1) * plane + 4 * c);
#pragma unroll
    for (int k = 0; k < 4; ++k) t = fmaf((float)((int)((w[i] >> (4 * k)) & 15u) - 8), xa[k], t);
#pragma unroll
    for (int k = 0; k < 4; ++k) t = fmaf((float)((int)((w[i] >> (4 * k + 16)) & 15u) - 8), xb[k], t);
  }
  return fmaf(sc, t, acc);
}

// ------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over the workgroup in a fixed order; every thread gets the result.
// `red` holds at least NT/64 floats of LDS.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) t += red[i];
  return t;
}

// Exclusive prefix sum of one int per thread over the workgroup (thread order).
// `red` holds at least NT/64 + 1 ints of LDS. Returns the exclusive prefix; the
// total goes to *total.
template <int NT>
__device__ __forceinline__ int block_excl_scan(int v, int* red, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int n = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += n;
  }
  __syncthreads();
  if (lane == 63) red[w] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) {
    if (i < w) base += red[i];
    tot += red[i];
  }
  *total = tot;
  return base + inc - v;
}

// Staging of an fp32 input vector x[d] (16-byte aligned, d % 4 == 0) into LDS (xs,
// fp32, in the layout of xs_index<T>); with LN (compile time) layer norm with gamma g and beta b (NULL: 0) is
// applied. load() only issues the global reads of x (then g and b) into registers, so
// that a caller can issue its own (HBM) loads behind them and still wait for these
// alone: the reads are not predicated per lane (index clamped, surplus lanes masked
// where used) and form straight-line code, which keeps the wait counts exact.
// finish() takes mean and biased variance as two workgroup reductions over the
// registers (two-pass, no cancellation), writes LDS and ends with a barrier.
// K float4 per thread covers d <= 4 * NT * K.
template <typename T, int NT, int K = (16384 / 4 + NT - 1) / NT, bool LN = false>
struct StageX {
  f32x4 v[K], gv[LN ? K : 1], bv[LN ? K : 1];
  __device__ __forceinline__ void load(const float* __restrict__ x, int d, const float* __restrict__ g,
                                       const float* __restrict__ b) {
    const int n4 = d >> 2;
#pragma unroll
    for (int k = 0; k < K; ++k)
      v[k] = *reinterpret_cast<const f32x4*>(x + 4 * min((int)threadIdx.x + k * NT, n4 - 1));
    if constexpr (LN) {
      const float* bp = b != nullptr ? b : g;   // a missing beta reads gamma, unused
#pragma unroll
      for (int k = 0; k < K; ++k)
        gv[k] = *reinterpret_cast<const f32x4*>(g + 4 * min((int)threadIdx.x + k * NT, n4 - 1));
#pragma unroll
      for (int k = 0; k < K; ++k)
        bv[k] = *reinterpret_cast<const f32x4*>(bp + 4 * min((int)threadIdx.x + k * NT, n4 - 1));
    }
  }
  __device__ __forceinline__ void finish(int d, bool has_b, float eps, float* xs, float* red) {
    const int n4 = d >> 2;
    // Surplus lanes (index clamped to n4 - 1) hold the last chunk's values and store
    // them to the same place as its own lane, so the stores need no predicate either.
    if constexpr (!LN) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int i = min((int)threadIdx.x + k * NT, n4 - 1);
        *reinterpret_cast<f32x4*>(xs + xs_index<T>(4 * i, d)) = v[k];
      }
      __syncthreads();
    } else {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < K; ++k)
        if ((int)threadIdx.x + k * NT < n4) s += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
      const float mean = block_sum<NT>(s, red) / (float)d;
      float q = 0.f;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if ((int)threadIdx.x + k * NT < n4) {
          const float a0 = v[k][0] - mean, a1 = v[k][1] - mean, a2 = v[k][2] - mean, a3 = v[k][3] - mean;
          q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
        }
      }
      const float rstd = 1.0f / sqrtf(block_sum<NT>(q, red) / (float)d + eps);
      const float bm = has_b ? 1.f : 0.f;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int i = min((int)threadIdx.x + k * NT, n4 - 1);
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (v[k][e] - mean) * rstd * gv[k][e] + bm * bv[k][e];
        *reinterpret_cast<f32x4*>(xs + xs_index<T>(4 * i, d)) = o;
      }
      __syncthreads();
    }
  }
};

// Stage a short vector x[d] (16-byte aligned, d % 4 == 0) into LDS as is, one
// predicated float4 per thread and step, then a barrier.
template <typename T, int NT>
__device__ void stage_x(const float* __restrict__ x, int d, float* xs) {
  for (int i = threadIdx.x; i < (d >> 2); i += NT)
    *reinterpret_cast<f32x4*>(xs + xs_index<T>(4 * i, d)) = *reinterpret_cast<const f32x4*>(x + 4 * i);
  __syncthreads();
}

// Order-preserving key of a float: a > b  <=>  key(a) > key(b); -0 maps to +0.
__device__ __forceinline__ uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ------------------------------------------------------------------ host
struct Workspace {
  size_t off = 0;
  char* base = nullptr;
  explicit Workspace(void* b) : base(static_cast<char*>(b)) {}
  template <typename P>
  P* take(size_t bytes) {
    P* p = reinterpret_cast<P*>(base ? base + off : nullptr);
    off += (bytes + 255) & ~size_t(255);
    return p;
  }
};

inline int elem_bytes(int dtype) { return dtype == DV_F16 ? 2 : 4; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int device_cu_count();   // cached per device

// Optional per-launch event recording (dv_set_launch_events), per calling thread.
void trace_reset();
void trace_begin(const char* label, hipStream_t st);
void trace_end(hipStream_t st);
// Events for the next kernel of an armed launch (both NULL when none is armed): the
// first kernel of the launch takes the start event, every kernel the end event.
void trace_take(hipEvent_t* start, hipEvent_t* stop);

// Every kernel goes through here. With events armed they are stamped by the kernel's
// own dispatch (hipExtLaunchKernel: its start and end times), not by separate marker
// commands around it, whose completion adds the queue's dispatch latency to the
// interval. Errors are left for hipGetLastError, as with a <<<>>> launch.
template <typename... P, typename... A>
inline void launch_k(void (*kern)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t st, A... args) {
  static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
  std::tuple<P...> vals(static_cast<P>(args)...);
  void* argv[sizeof...(P) + 1];
  std::apply([&argv](auto&... v) {
    int i = 0;
    ((argv[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  trace_take(&e0, &e1);
  const void* f = reinterpret_cast<const void*>(kern);
  if (e1 != nullptr) (void)hipExtLaunchKernel(f, grid, block, argv, lds, st, e0, e1, 0);
  else (void)hipLaunchKernel(f, grid, block, argv, lds, st);
}

#define DV_LAUNCH(label, stream, expr)              \
  do {                                              \
    ::dv::trace_begin(label, stream);               \
    const hipError_t dv_e_ = (expr);                \
    ::dv::trace_end(stream);                        \
    if (dv_e_ != hipSuccess) return DV_ERR_HIP;     \
  } while (0)

// ---------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error. All work goes on `st`.

// Select per row of scores [B][n]: top-k or threshold, ascending output.
hipError_t launch_select(const float* scores, int B, int n, int mode, int k, float thresh,
                         int32_t* idx, int cap, int32_t* count, int32_t* idx2, hipStream_t st);

// Device-side check that each of B sets set[b][0..n) is strictly ascending within
// [0, range); writes 0 (valid) or 1 to *bad.
hipError_t launch_validate_sets(const int32_t* set, int B, int n, int range, int32_t* bad, hipStream_t st);

// Predictor hidden layer: hid[b][j] = x-hat[b] . AT[j], for up to two predictors
// sharing one input (rows of P0 first, then rows of P1). LN applied if g != NULL.
struct PredHidArgs {
  int d, B;
  const float* x;           // [B][d]
  const float* g; const float* be; float eps;
  const void* AT0; int r0; float* hid0;   // [B][r0]
  const void* AT1; int r1; float* hid1;   // [B][r1] (r1 = 0: none)
  float* xhat_out;                        // optional [B][d]: the normalised input, written once
};
hipError_t launch_pred_hidden(int wtype, const PredHidArgs& a, hipStream_t st);

// Predictor scores: s[b][i] = hid[b] . BT[i] for up to two predictors.
struct PredScoreArgs {
  int r0, n0; const void* BT0; const float* hid0; float* s0;   // hid0 [B][r0], s0 [B][n0]
  int r1, n1; const void* BT1; const float* hid1; float* s1;   // n1 = 0: none
  int B;
  // sel_k0 > 0 (B = 1, n0 <= workgroup size): one extra workgroup computes all n0
  // scores of the first predictor and writes their top-sel_k0 set, ascending, to
  // sel_set0 (and sel_set0_out if not NULL).
  int sel_k0; int32_t* sel_set0; int32_t* sel_set0_out;
};
hipError_t launch_pred_scores(int wtype, const PredScoreArgs& a, hipStream_t st);

// Gathered row-dot for Q/K/V of the selected heads (B = 1).
struct QkvArgs {
  int d, H, dh, cap, pos, n_heads;
  const float* x;                   // input (layer-normalised here if g is set)
  const float* g; const float* be; float eps;   // optional LN of x inside the launch (g NULL: none)
  const void* Wq; const void* Wk; const void* Wv;
  const float* bq; const float* bk; const float* bv;
  void* K; void* V;                 // [H][cap][dh] of this sequence
  float* q;                         // [n_heads][dh] out
  const int32_t* heads_in;          // [n_heads] the head set
  int32_t* heads_ws;                // optional [n_heads] out: the set, clamped (one workgroup)
  uint8_t* valid;                   // optional [H][cap]: row pos marked present for the set, absent otherwise
  // Top-k selection run by one extra workgroup of the launch (sel_n == 0: none).
  const float* sel_scores; int sel_n; int sel_k; int32_t* sel_idx; int32_t* sel_idx_out;
  uint32_t* clear; int clear_n;     // counters of a later row-axpy to zero (optional)
  // Rows of up to two more matrices of the weights' type dotted with the same input
  // after the Q/K/V rows (the next layer's predictor first layers, which read this
  // layer's normalised input): hid0[j] = x-hat . AT0[j] (j < r0), likewise AT1 (r0, r1 = 0: none).
  const void* AT0; int r0; float* hid0;
  const void* AT1; int r1; float* hid1;
  // The missing-KV fill's listing run by one extra workgroup instead (list NULL: none;
  // not with a hosted selection): for each selected head j, the positions below pos
  // marked 0 in valid, ascending, in list[j * list_stride ..], their count in list_count[j].
  int32_t* list; int list_stride; int32_t* list_count;
};
hipError_t launch_qkv(int wtype, int kvtype, const QkvArgs& a, hipStream_t st);

// Largest batch of the batched (matrix-core) path: token columns of one MFMA tile pair.
constexpr int kMaxBatch = 32;

// Split-KV decode attention for the selected heads of B sequences (grid z = sequence).
struct AttnArgs {
  int H, dh, cap, n_heads, n_split, chunk;
  int posb[kMaxBatch];              // row of the current token, per sequence
  // reorder != 0: grid slot z (blockIdx.z) attends sequence seq_of[z] (a permutation of
  // the batch), so that the host can choose which workgroups share a CU.
  int seq_of[kMaxBatch];
  int reorder;
  const float* q;                   // [B][n_heads][dh]
  const int32_t* heads;             // [B][n_heads]
  const void* K; const void* V;     // [B][H][cap][dh]
  float scale;
  float* part;                      // [B][n_heads][n_split][dh + 2]
  // One chunk per head (n_split == 1) and C set: the output H_h(x_b) goes straight to
  // the out-projection's fp16 coefficients C(b, p * dh + t) (p: h's place in the union
  // list ulist[0..*ucount)) instead of a partial; the rest of C is zeroed beforehand.
  _Float16* C; int ldc; int cnb; const int32_t* ulist; const int32_t* ucount;   // C: coef_index layout, cnb tokens
  uint8_t* valid;                   // optional [B][H][cap]: rows attended are marked present
};
hipError_t launch_attn(int kvtype, const AttnArgs& a, int B, hipStream_t st);

// Missing keys and values (B = 1): for every selected head, the cache rows t < pos
// whose valid[h][t] is 0 are computed from the kept inputs Y[t] (K[h][t] = Y[t] . W^K_h
// rows + bk, likewise V); Y[pos] = x is kept for later tokens. The valid marks are set
// by the launches that follow (QKV at pos, attention over 0..pos), never here.
struct KvFillArgs {
  int d, H, dh, cap, pos, n_heads;
  const float* x;                   // [d] this token's attention input
  void* Y;                          // [cap][d] kept attention inputs, in the cache's type
  const uint8_t* valid;             // [H][cap]
  const int32_t* heads;             // [n_heads]
  const void* Wk; const void* Wv; const float* bk; const float* bv;
  void* K; void* V;                 // [H][cap][dh]
};
hipError_t launch_kv_fill(int wtype, int kvtype, const KvFillArgs& a, hipStream_t st);
// The fill after a QKV launch that listed each selected head's missing positions
// (ascending) in list[j * stride ..] (stride >= pos) and their count in
// list[n_heads * stride + j]: a resident grid streams the listed heads' rows, and
// keeps this token's input.
hipError_t launch_kv_fill_listed(int wtype, int kvtype, const KvFillArgs& a, const int32_t* list, int stride,
                                 hipStream_t st);
// Y[pos] = x in the cache's type alone (no head selected, so no fill runs).
hipError_t launch_keep_input(int kvtype, const KvFillArgs& a, hipStream_t st);

// Gathered row-axpy: out = resid + bias + sum_rows coef[row] * M[rowidx(row)], tiled by
// 128-byte column tiles; every workgroup sums all selected rows of its tile.
struct AxpyArgs {
  int d, nrows;                     // row length, selected rows
  const void* M; int m_rows;        // M is [m_rows][d]
  // Row source: neuron rows (rows = set) or head rows (rows = set[row / dh] * dh + row % dh).
  const int32_t* set; int dh;       // dh = 0: neuron rows
  // Coefficients: coef[row] (neurons), or from attention partials (heads).
  const float* coef;
  const _Float16* scales;           // 4-bit rows only: [m_rows][d / 32] chunk scales
  const float* part; int n_split;   // attention partials when coef == NULL
  const float* resid; const float* bias;   // optional, [d]
  float* out;                        // [d]
  float* out2;                       // optional second copy of out
  // Row-split partial sums [kAxpyMaxRowSplit][d] (workspace); NULL: one split.
  float* partial;
  // Per column span arrival counters [kAxpyMaxSpans], zero at launch (an earlier
  // kernel of the same call clears them): the last split of a span to arrive adds
  // the partials. NULL: a second launch adds them.
  uint32_t* cnt;
  int rows_per_batch;                // set by the launcher
};
constexpr int kAxpyMaxRowSplit = 32;
constexpr int kAxpyMaxSpans = 64;     // column spans of 64 x 16 bytes at d <= 16000

// Raises a kernel's dynamic LDS limit on the current device when a launch needs more
// than the 64 KB default. The limit set is always the same for a kernel and device (the
// device's LDS per workgroup less the kernel's static LDS), so concurrent callers
// agree; which (kernel, device) pairs are done is kept in a mutex-guarded set. A
// request above that limit returns hipErrorInvalidValue.
hipError_t ensure_dyn_lds(const void* kern, size_t bytes);
int device_lds_per_block();   // cached per device

// Clears n counters for a later row-axpy of the same call (agent-scope stores: the
// counters are read by atomics from every XCD).
__device__ __forceinline__ void clear_counters(uint32_t* c, int n) {
  if (c != nullptr && blockIdx.x == 0)
    for (int i = threadIdx.x; i < n; i += blockDim.x) __hip_atomic_store(c + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
hipError_t launch_axpy(int wtype, const AxpyArgs& a, hipStream_t st);

// fc1 + ReLU over the selected neurons (B = 1): h[s] = max(x-hat . W1T[set[s]] + b1, 0).
struct Fc1Args {
  int d, k, n;                      // width, selected neurons, neurons in W1T
  const float* x; const float* g; const float* be; float eps;    // LN (g NULL: none)
  const void* W1T; const float* b1; const int32_t* set;
  const _Float16* s1;               // 4-bit rows only: [n][d / 32] chunk scales
  int act;                          // kActRelu / kActGelu
  float* h;
  uint32_t* clear; int clear_n;     // counters of a later row-axpy to zero (optional)
};
hipError_t launch_fc1(int wtype, const Fc1Args& a, hipStream_t st);

// ------------------------------------------------ batched (matrix-core) path
// Union of B ascending sets in [0, n): U ascending, *count and optional membership
// bits mask[u] (bit b: U[u] is in set b). Needs union_lds_bytes(n) of LDS per
// workgroup (no scratch memory).
size_t union_lds_bytes(int n);
hipError_t launch_union(const int32_t* sets, int B, int k, int n, int32_t* U, int32_t* count, uint32_t* mask,
                        hipStream_t st);

// X16[NB][Kpad] = fp16(LN(x)) (g NULL: x), zero rows b >= B and columns k >= d.
hipError_t launch_ln_cast(const float* x, int B, int NB, int d, int Kpad, const float* g, const float* be, float eps,
                          _Float16* X16, hipStream_t st);
// The cast above and the union of the B sets (launch_union) in one launch.
hipError_t launch_cast_union(const float* x, int B, int NB, int d, int Kpad, const float* g, const float* be,
                             float eps, _Float16* X16, const int32_t* sets, int k, int n, int32_t* U,
                             int32_t* count, uint32_t* mask, hipStream_t st);

enum { kRowsList = 0, kRowsHeads = 1, kRowsIdentity = 2 };

// Gathered rows times the token batch on the matrix cores, split over K:
// P[s][r][b] = sum_{k in split s} W(r)[k] X16[b][k]. Rows: kRowsList W0[list[r]];
// kRowsHeads r = (m * nu + p) * dh + t -> row list[p] * dh + t of W0/W1/W2 (m = 0, 1, 2);
// kRowsIdentity r < n0 -> W0[r], else W1[r - n0]. With out0 set (and S == 1) the
// result goes straight to out0[b][r] (r < n0) / out1[b][r - n0] for b < B.
struct MrowsArgs {
  int d, Kpad, Ks, S;
  const _Float16* X;                 // [NB][Kpad]
  int mode;
  const void* W0; const void* W1; const void* W2;   // fp16 rows of d elements
  const int32_t* list; const int32_t* list_count; int list_max; int dh;
  int list_range;                    // list entries are clamped to [0, list_range)
  int nrows, n0;                     // kRowsIdentity: rows in all, rows of W0
  float* P; int nrows_pad;           // [S][nrows_pad][NB]
  float* out0; int ld0; float* out1; int ld1; int B;
};
void mrows_split(int Kpad, int NB, int* S, int* Ks);
hipError_t launch_mrows(int NB, const MrowsArgs& a, hipStream_t st);

// Token-batch coefficients times gathered rows, contracted over the rows:
// P[s][b][c] = sum_{u in split s} C(b, u) M[row(u)][c], row(u) = list[u] (dh == 0) or
// list[u / dh] * dh + u % dh. C is fp16, NB tokens x ldc rows (ldc a multiple of 32) in the
// blocked layout of coef_index, zero beyond the rows in use.
struct McolsArgs {
  int d;
  const void* M;
  const int32_t* list; const int32_t* list_count; int list_max; int dh;
  int list_range;                    // list entries are clamped to [0, list_range)
  const _Float16* C; int ldc;
  int S, B;
  float* P;                          // [S][B][d]
};
int mcols_split(int d, int nmax);
hipError_t launch_mcols(int NB, const McolsArgs& a, hipStream_t st);

// Coefficient matrices of the contraction over gathered rows (k_mfma_cols' C): blocks of 32
// rows, each NB tokens x 32 rows row-major, so that the 32 rows one k-step contracts are
// one contiguous NB * 64-byte piece (a wavefront's coefficient load then covers whole
// 128-byte lines instead of 64-byte pieces of 16 token rows).
__host__ __device__ __forceinline__ size_t coef_index(int b, int u, int nb) {
  return ((size_t)(u >> 5) * nb + b) * 32 + (u & 31);
}

// C(b, u) = fp16(sigma(sum_s P[s][u][b] + b1[list[u]])), masked by membership bits
// (C in the layout of coef_index).
struct Fc1FinishArgs {
  const float* P; int S, nrows_pad;
  const int32_t* list; const int32_t* list_count; int list_max; int list_range;
  const float* b1; const uint32_t* mask; int B; int act;
  _Float16* C; int ldc;
};
hipError_t launch_fc1_finish(int NB, const Fc1FinishArgs& a, hipStream_t st);

// out[b][c] = sum_s P[s][b][c] + bias[c] + resid[b][c].
struct ColsFinishArgs {
  const float* P; int S, B, d;
  const float* bias; const float* resid; float* out;
};
hipError_t launch_cols_finish(const ColsFinishArgs& a, hipStream_t st);

// C[b][j] = fp16(sum_s P[s][row0 + j][b]) for j < r, zero padded to [NB][ldc].
hipError_t launch_sum_cast(int NB, const float* P, int S, int nrows_pad, int row0, int r, int B, _Float16* C, int ldc,
                           hipStream_t st);

// Q/K/V from kRowsHeads partials: q[b][j][t] and cache rows pos[b] of the selected heads.
struct QkvFinishArgs {
  const float* P; int S, nrows_pad;
  const int32_t* heads; int n_heads, H, dh, cap, B;
  const int32_t* hlist; const int32_t* hcount;     // union of the head sets and its size
  const float* bq; const float* bk; const float* bv;
  float* q; void* K; void* V;
  int posb[kMaxBatch];
  _Float16* zero; int zero_n;       // optional: halves to clear (multiple of 8, 16-byte aligned)
};
hipError_t launch_qkv_finish(int NB, int kvtype, const QkvFinishArgs& a, hipStream_t st);

// Out-projection coefficients C(b, p*dh + t) (coef_index layout) from the split-KV partials.
struct AttnFinishArgs {
  const float* part; int n_split, n_heads, dh, B;
  const int32_t* heads; const int32_t* list; const int32_t* hcount;
  _Float16* C; int ldc;
};
hipError_t launch_attn_finish(int NB, const AttnFinishArgs& a, hipStream_t st);

// Host side of the batched path (dv_batch_api.hip); arguments already validated.
int batch_nb(int B);
int batch_max_rank(int B);
size_t batch_mlp_ws(const dv_mlp* m, int B, int n_idx, int per_seq);
size_t batch_attn_ws(const dv_attn* a, int B, int n_heads);
size_t batch_block_ws(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa, const dv_predictor* pm, int B,
                      int kh, int km);
dv_status batch_mlp(const dv_mlp* m, const float* x, int B, const int32_t* idx, int n_idx, int per_seq,
                    int batch_mode, float* out, void* ws, size_t ws_bytes, uint32_t flags, hipStream_t hs);
dv_status batch_attn(const dv_attn* a, const float* x, int B, const dv_kv* kv, const int32_t* heads, int n_heads,
                     float scale, float* out, void* ws, size_t ws_bytes, uint32_t flags, hipStream_t hs);
dv_status batch_block(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa, const dv_predictor* pm,
                      const dv_ln* ln, const dv_kv* kv, const float* x_in, float* x_out, int B, int kh, int km,
                      int mode, int batch_mode, float scale, int32_t* heads_out, int32_t* idx_out, void* ws,
                      size_t ws_bytes, hipStream_t hs);
// DV_VALIDATE: check B ascending sets of n indices in [0, range) (synchronises `st`).
dv_status validate_sets_sync(const int32_t* set, int B, int n, int range, int32_t* flag, hipStream_t st);

// Host-side argument checks shared by the entry points (dv_api.hip).
constexpr int kMaxWidth = 16000;   // widest row the row-dot kernels stage in LDS
bool dtype_ok(int t);
int chunk_elems(int t);            // elements per 16-byte chunk
bool ws_ok(void* ws);              // non-NULL and 256-byte aligned
dv_status check_mlp(const dv_mlp* m);
dv_status check_attn(const dv_attn* a);
dv_status check_kv(const dv_kv* kv, const dv_attn* a, int B);
dv_status check_ln(const dv_ln* ln);
dv_status check_predictor_for(const dv_predictor* p, int d, int n_out);
size_t axpy_partial_bytes(int d);  // row-split partial sums of a row-axpy of width d

// Split-KV chunk length (positions per attention workgroup); at most kAttnMaxSplit
// chunks per head.
constexpr int kAttnMaxSplit = 16;
int attn_chunk(int n_heads, int attended, int dh, int kvtype);

}  // namespace dv
