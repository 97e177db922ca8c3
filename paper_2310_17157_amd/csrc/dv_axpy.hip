// Gathered row-axpy: out = resid + bias + sum_rows coef[row] * M[rowidx(row), :].
//
// This is the second half of both sparsified blocks: the MLP's
// sum_{i in S_M} ReLU(z_i) W^2_i over rows of W2T (Eq. (1)), and the attention's
// sum_{i in S_A} H_i(y) W^O_i over the dh rows of each selected head in WoT (Eq. (2)).
// Both weights are stored transposed so that a selected neuron or head is a set of
// whole contiguous rows (Section 4.4 "Memory coalescing").
//
// Tiling: the grid is (column spans) x (row splits). A span is 64 lanes x 16 bytes,
// so every wavefront load instruction reads 1 KB of one row, contiguous in memory;
// workgroup (c, s) sums span c of the rows in split s, wavefront w taking the rows
// w, w + NW, ... of the split with U loads in flight and the next U issued before the
// current are consumed. Wavefront partials are added in LDS in wavefront order; with
// one split the workgroup writes out directly, otherwise it writes its partial row
// to partial[s], and the splits are added in split order (bitwise reproducible) by
// either a second small launch or, given arrival counters, the last split of each
// span to arrive. The counter protocol needs no fence that writes back or
// invalidates a whole L2: partials are written and read with agent-scope (coherent,
// L2-bypassing) atomic stores and loads, each workgroup waits for its stores to be
// acknowledged before it increments its span's counter, and the workgroup that
// draws the last ticket reads every split after that. The HIP memory model alone does
// not order relaxed atomics on different addresses; the protocol rests on gfx950
// compiling agent-scope stores and loads to sc1 accesses (write-through to, and reads
// from, the memory side shared by all XCDs), on s_waitcnt returning only once those
// stores are acknowledged, and on the barrier that follows (also a compiler barrier)
// keeping the ticket below every wavefront's wait.
//
// For the attention the coefficients H_i(y)[t] are combined first, in the prologue,
// from the split-KV partials (max logit, sum of exponentials and unnormalised value
// sums per position chunk) of the heads of the workgroup's rows, while the first
// weight loads are in flight.
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

constexpr int kAxNW = 8;    // wavefronts per workgroup
constexpr int kAxU = 8;     // row loads per batch (two batches in flight)
constexpr int kAxRowsLds = 3072;   // (coefficient, row index) pairs per LDS batch

constexpr int kAxMaxSplit = kAttnMaxSplit;   // split-KV chunks, combined with all loads in flight

// HEADS selects the attention form (rows are dh-row blocks of selected heads, the
// coefficients are combined from split-KV partials); otherwise rows are single
// neurons with coefficients given per row. R rows share one load instruction, each
// read by 64 / R lanes (R = 4 for 4-bit rows, whose 16-byte chunk holds 32 columns:
// a span stays 512 columns wide, as for fp16 rows).
template <typename T, int NW, int U, bool HEADS, int R = 1>
__global__ void __launch_bounds__(NW * 64) k_axpy(AxpyArgs a) {
  constexpr int NT = NW * 64;
  constexpr int E = Chunk<T>::E;
  constexpr int LR = 64 / R;                                     // lanes per row of a load
  constexpr int SW = LR * E;                                     // columns per span
  extern __shared__ float smem[];
  const int rpb = a.rows_per_batch;
  float* cf = smem;                                              // [rpb] coefficients
  int* ri = reinterpret_cast<int*>(cf + rpb);                    // [rpb] row indices
  float* red = reinterpret_cast<float*>(ri + rpb);               // [NW][SW] wavefront sums
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int q = R == 1 ? 0 : lane / LR, lcol = lane - q * LR;   // row of a load, lane within the row
  const int S = gridDim.y, sp = blockIdx.y;
  const int r0 = (int)((long)sp * a.nrows / S), r1 = (int)((long)(sp + 1) * a.nrows / S);
  constexpr bool Q4 = kIsQ4<T>;
  const int nch = a.d / E;
  const int lc = min((int)blockIdx.x * LR + lcol, nch - 1);          // this lane's chunk of a row
  const char* Mb = static_cast<const char*>(a.M) + (size_t)lc * 16;
  const size_t rowb = Q4 ? (size_t)a.d / 2 : (size_t)a.d * sizeof(T);
  const _Float16* Sb = Q4 ? a.scales + lc : nullptr;                  // 4-bit rows: chunk scales
  const int srow = a.d / 32;
  const int ns = a.n_split;
  const int stride = a.dh + 2;

  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;

  for (int rb = r0; rb < r1; rb += rpb) {
    const int nb = min(rpb, r1 - rb);
    // ---- row indices (they need only the set), then this wavefront's first loads
    for (int i = tid; i < nb; i += NT) {
      const int row = rb + i;
      if (!HEADS) {
        ri[i] = min(max(a.set[row], 0), a.m_rows - 1);
      } else {
        const int h = row / a.dh;
        ri[i] = min(max(a.set[h], 0), a.m_rows / a.dh - 1) * a.dh + (row - h * a.dh);
      }
    }
    __syncthreads();
    // this wavefront's groups of R rows: wave + NW * i, i < nwr; loads past the end are
    // clamped to the last row (and weighted by zero), so every batch issues U loads
    const int ng = (nb + R - 1) / R;
    const int nwr = ng > wave ? (ng - wave + NW - 1) / NW : 0;
    struct Batch {
      u32x4 w[U];
      _Float16 s[Q4 ? U : 1];
    };
    auto load = [&](Batch& b, int i0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = min((wave + NW * (i0 + u)) * R + q, nb - 1);
        b.w[u] = ld_stream(Mb + (size_t)ri[i] * rowb);
        if constexpr (Q4) b.s[u] = Sb[(size_t)ri[i] * srow];
      }
    };
    auto consume = [&](const Batch& b, int i0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u, row = (wave + NW * i) * R + q;
        float f = i < nwr && (R == 1 || row < nb) ? cf[row] : 0.f;
        if constexpr (Q4) f *= (float)b.s[u];
        float v[E];
        unpack<T>(b.w[u], v);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(f, v[e], acc[e]);
      }
    };
    Batch wa, wb;
    if (nwr > 0) load(wa, 0);
    // ---- coefficients, while those loads are in flight
    if (!HEADS) {
      for (int i = tid; i < nb; i += NT) cf[i] = a.coef[rb + i];
    } else {
      // one thread per row reads its head's (m_s, l_s) and its own o_s[t] of every
      // chunk s in one round: H(y)[t] = sum_s e^{m_s - M} o_s[t] / sum_s e^{m_s - M} l_s
      for (int i = tid; i < nb; i += NT) {
        const int row = rb + i;
        const int h = row / a.dh, t = row - h * a.dh;
        const float* P = a.part + (size_t)h * ns * stride;
        float m[kAxMaxSplit], l[kAxMaxSplit], o[kAxMaxSplit];
#pragma unroll
        for (int s = 0; s < kAxMaxSplit; ++s) {
          m[s] = s < ns ? P[(size_t)s * stride] : -INFINITY;
          l[s] = s < ns ? P[(size_t)s * stride + 1] : 0.f;
          o[s] = s < ns ? P[(size_t)s * stride + 2 + t] : 0.f;
        }
        float M = -INFINITY;
#pragma unroll
        for (int s = 0; s < kAxMaxSplit; ++s) M = fmaxf(M, m[s]);
        float L = 0.f, num = 0.f;
#pragma unroll
        for (int s = 0; s < kAxMaxSplit; ++s) {
          const float f = m[s] == -INFINITY ? 0.f : __expf(m[s] - M);
          L = fmaf(l[s], f, L);
          num = fmaf(o[s], f, num);
        }
        cf[i] = num / L;
      }
    }
    __syncthreads();

    // ---- stream, alternating two register sets
    if (nwr > 0) {
      for (int i0 = 0;;) {
        if (i0 + U < nwr) load(wb, i0 + U);
        consume(wa, i0);
        i0 += U;
        if (i0 >= nwr) break;
        if (i0 + U < nwr) load(wa, i0 + U);
        consume(wb, i0);
        i0 += U;
        if (i0 >= nwr) break;
      }
    }
    __syncthreads();   // ri / cf are rewritten by the next batch
  }
  // ---- combine the R rows of a load (lanes q and q ^ 1, then q and q ^ 2, ...),
  // then wavefronts in order, then write out (one split) or partial[sp]
#pragma unroll
  for (int off = LR; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += __shfl_xor(acc[e], off);
  if (q == 0)
#pragma unroll
    for (int e = 0; e < E; ++e) red[wave * SW + lcol * E + e] = acc[e];
  __syncthreads();
  for (int t = tid; t < SW; t += NT) {
    const int col = blockIdx.x * SW + t;
    if (col < a.d) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w * SW + t];
      if (S == 1) {
        if (a.resid) s += a.resid[col];
        if (a.bias) s += a.bias[col];
        a.out[col] = s;
        if (a.out2) a.out2[col] = s;
      } else if (a.cnt == nullptr) {
        a.partial[(size_t)sp * a.d + col] = s;
      } else {
        __hip_atomic_store(a.partial + (size_t)sp * a.d + col, s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (S == 1 || a.cnt == nullptr) return;
  // ---- arrival: stores acknowledged, then one ticket per workgroup; the last adds
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  __shared__ int last;
  if (tid == 0)
    last = __hip_atomic_fetch_add(a.cnt + blockIdx.x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)(S - 1);
  __syncthreads();
  if (!last) return;
  for (int t = tid; t < SW; t += NT) {
    const int col = blockIdx.x * SW + t;
    if (col < a.d) {
      float p[kAxpyMaxRowSplit];
#pragma unroll
      for (int s = 0; s < kAxpyMaxRowSplit; ++s)
        if (s < S) p[s] = __hip_atomic_load(a.partial + (size_t)s * a.d + col, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      float v = p[0];
#pragma unroll
      for (int s = 1; s < kAxpyMaxRowSplit; ++s)
        if (s < S) v += p[s];
      if (a.resid) v += a.resid[col];
      if (a.bias) v += a.bias[col];
      a.out[col] = v;
      if (a.out2) a.out2[col] = v;
    }
  }
  if (tid == 0) __hip_atomic_store(a.cnt + blockIdx.x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// out = sum_s partial[s] (in split order) + resid + bias; four columns per thread,
// every split's load issued before the first add.
__global__ void __launch_bounds__(256) k_axpy_sum(AxpyArgs a, int S) {
  const int i = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= a.d) return;
  f32x4 p[kAxpyMaxRowSplit];
#pragma unroll
  for (int s = 0; s < kAxpyMaxRowSplit; ++s)
    if (s < S) p[s] = *reinterpret_cast<const f32x4*>(a.partial + (size_t)s * a.d + i);
  f32x4 v = p[0];
#pragma unroll
  for (int s = 1; s < kAxpyMaxRowSplit; ++s)
    if (s < S) v += p[s];
  if (a.resid) v += *reinterpret_cast<const f32x4*>(a.resid + i);
  if (a.bias) v += *reinterpret_cast<const f32x4*>(a.bias + i);
  *reinterpret_cast<f32x4*>(a.out + i) = v;
  if (a.out2) *reinterpret_cast<f32x4*>(a.out2 + i) = v;
}

// Row splits: enough workgroups to give every CU one, each split at least two groups
// of rows per wavefront; one split when there is no partial buffer.
static int axpy_row_splits(int spans, int nrows, int rows_per_round) {
  int S = device_cu_count() / spans;
  S = min(S, nrows / (2 * rows_per_round));
  return max(1, min(S, kAxpyMaxRowSplit));
}

template <typename T, bool HEADS, int NW = kAxNW, int U = kAxU, int R = 1>
static hipError_t launch_axpy_t(AxpyArgs a, hipStream_t st) {
  constexpr int E = Chunk<T>::E;
  constexpr int LR = 64 / R;
  const int spans = (a.d / E + LR - 1) / LR;
  const int S = a.partial != nullptr ? axpy_row_splits(spans, a.nrows, NW * R) : 1;
  if (spans > kAxpyMaxSpans) a.cnt = nullptr;   // no counter per span: the split sum is a launch
  // LDS: (coefficient, row index) pairs of a batch of the split's rows and the
  // wavefront sums.
  const int rpb = min(kAxRowsLds, max(1, (a.nrows + S - 1) / S));
  a.rows_per_batch = rpb;
  const size_t lds = (size_t)rpb * 8 + (size_t)NW * LR * E * 4;
  launch_k((k_axpy<T, NW, U, HEADS, R>), dim3(spans, S), dim3(NW * 64), lds, st, a);
  if (S > 1 && a.cnt == nullptr) launch_k(k_axpy_sum, dim3((a.d / 4 + 255) / 256), dim3(256), 0, st, a, S);
  return hipGetLastError();
}

hipError_t launch_axpy(int wtype, const AxpyArgs& a, hipStream_t st) {
  // 4-bit rows: 32 columns per lane, so a load covers 4 rows of a 512-column span;
  // 8 wavefronts with batches of 2 loads (19.0 -> 13.9-14.4 us at the OPT-175B set
  // against the 2048-column spans of one row per load with a separate split-sum
  // launch; batches of 4 and 8, and 4 wavefronts, were slower)
  if (wtype == DV_Q4) return a.dh > 0 ? hipErrorInvalidValue : launch_axpy_t<q4_t, false, 8, 2, 4>(a, st);
  if (a.dh > 0)
    return wtype == DV_F16 ? launch_axpy_t<_Float16, true>(a, st) : launch_axpy_t<float, true>(a, st);
  return wtype == DV_F16 ? launch_axpy_t<_Float16, false>(a, st) : launch_axpy_t<float, false>(a, st);
}

}  // namespace dv
