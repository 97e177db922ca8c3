// Gathered row-axpy: out = resid + bias + sum_rows coef[row] * M[rowidx(row), :].
//
// This is the second half of both sparsified blocks: the MLP's
// sum_{i in S_M} ReLU(z_i) W^2_i over rows of W2T (Eq. (1)), and the attention's
// sum_{i in S_A} H_i(y) W^O_i over the dh rows of each selected head in WoT (Eq. (2)).
// Both weights are stored transposed so that a selected neuron or head is a set of
// whole contiguous rows (Section 4.4 "Memory coalescing").
//
// Tiling: a workgroup owns a 128-byte column tile (8 lanes x one 16-byte chunk) of
// every selected row, so each wavefront load instruction covers 8 rows and each
// wavefront keeps U such instructions in flight. The workgroup sums all selected rows
// of its tile, so no cross-workgroup reduction, atomics or device-scope fences are
// needed (on a multi-XCD part a device-scope release writes back the whole L2 of the
// XCD). Lane partials are combined across row groups with shuffles and across
// wavefronts in LDS, in a fixed order: the result is bitwise reproducible.
//
// For the attention the coefficients H_i(y)[t] are combined first, in the prologue,
// from the split-KV partials (max logit, sum of exponentials and unnormalised value
// sums per position chunk) of every selected head.
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

constexpr int kAxNW = 16;   // wavefronts per workgroup
constexpr int kAxTL = 8;    // lanes (16-byte chunks) per row segment: 128-byte tiles
constexpr int kAxU = 8;     // row instructions per batch (two batches in flight)

constexpr int kAxMaxSplit = kAttnMaxSplit;   // split-KV chunks, combined with all loads in flight

template <typename T, int TL, int U>
__device__ __forceinline__ void ax_load(u32x4 (&w)[U], const char* Mb, size_t rowb, const int* ri, int r,
                                        int step, int nb) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int row = r + step * u;
    w[u] = row < nb ? ld_stream(Mb + (size_t)ri[row] * rowb) : u32x4{0u, 0u, 0u, 0u};
  }
}

template <typename T, int E, int U>
__device__ __forceinline__ void ax_consume(const u32x4 (&w)[U], const float* cf, int r, int step, int nb,
                                           float (&acc)[E]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int row = r + step * u;
    float v[E];
    unpack<T>(w[u], v);
    const float f = row < nb ? cf[row] : 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = fmaf(f, v[e], acc[e]);
  }
}

// HEADS selects the attention form (rows are dh-row blocks of selected heads, the
// coefficients are combined from split-KV partials); otherwise rows are single
// neurons with coefficients given per row.
template <typename T, int NW, int TL, int U, bool HEADS>
__global__ void __launch_bounds__(NW * 64) k_axpy(AxpyArgs a) {
  constexpr int NT = NW * 64;
  extern __shared__ float smem[];
  constexpr int E = Chunk<T>::E;
  constexpr int RPI = 64 / TL;                  // rows per load instruction
  constexpr int step = NW * RPI;                // rows per wavefront-group step
  float* cf = smem;                                              // [rows_per_batch] coefficients
  int* ri = reinterpret_cast<int*>(cf + a.rows_per_batch);       // [rows_per_batch] row indices
  float* red = reinterpret_cast<float*>(ri + a.rows_per_batch);  // [NW][TL*E] wavefront sums
  float* fac = red + NW * TL * E;                                // [heads of a batch][n_split]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nch = a.d / E;
  const int c = blockIdx.x * TL + (lane % TL);
  const int grp = lane / TL;
  const bool on = c < nch;

  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  const char* Mb = static_cast<const char*>(a.M) + (size_t)(on ? c : 0) * 16;
  const size_t rowb = (size_t)a.d * sizeof(T);
  const int ns = a.n_split;
  const int stride = a.dh + 2;

  // Rows are processed in batches of at most rows_per_batch so that their
  // coefficients and row indices fit in LDS.
  for (int rb = 0; rb < a.nrows; rb += a.rows_per_batch) {
    const int nb = min(a.rows_per_batch, a.nrows - rb);
    const int h0 = HEADS ? rb / a.dh : 0;
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
    const int rfirst = wave * RPI + grp;
    u32x4 wa[U];
    if (on) ax_load<T, TL, U>(wa, Mb, rowb, ri, rfirst, step, nb);
    // ---- coefficients, while those loads are in flight
    if (!HEADS) {
      for (int i = tid; i < nb; i += NT) cf[i] = a.coef[rb + i];
    } else {
      // fac[h][s] = exp(m_s - M_h) / L_h for the heads of this batch (ns <= kAxMaxSplit)
      const int h1 = (rb + nb - 1) / a.dh;
      for (int hh = tid; hh <= h1 - h0; hh += NT) {
        const float* P = a.part + (size_t)(h0 + hh) * ns * stride;
        float m[kAxMaxSplit], l[kAxMaxSplit];
        float M = -INFINITY;
#pragma unroll
        for (int sp = 0; sp < kAxMaxSplit; ++sp) {
          m[sp] = sp < ns ? P[(size_t)sp * stride] : -INFINITY;
          l[sp] = sp < ns ? P[(size_t)sp * stride + 1] : 0.f;
          M = fmaxf(M, m[sp]);
        }
        float L = 0.f;
#pragma unroll
        for (int sp = 0; sp < kAxMaxSplit; ++sp) {
          m[sp] = m[sp] == -INFINITY ? 0.f : __expf(m[sp] - M);
          L += l[sp] * m[sp];
        }
        const float inv = 1.f / L;
#pragma unroll
        for (int sp = 0; sp < kAxMaxSplit; ++sp)
          if (sp < ns) fac[hh * ns + sp] = m[sp] * inv;
      }
      __syncthreads();
      for (int i = tid; i < nb; i += NT) {
        const int row = rb + i;
        const int h = row / a.dh, t = row - h * a.dh;
        const float* P = a.part + (size_t)h * ns * stride + 2 + t;
        const float* F = fac + (h - h0) * ns;
        float o[kAxMaxSplit];
#pragma unroll
        for (int sp = 0; sp < kAxMaxSplit; ++sp) o[sp] = sp < ns ? P[(size_t)sp * stride] : 0.f;
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int sp = 0; sp < kAxMaxSplit; sp += 2) {
          if (sp < ns) s0 = fmaf(o[sp], F[sp], s0);
          if (sp + 1 < ns) s1 = fmaf(o[sp + 1], F[sp + 1], s1);
        }
        cf[i] = s0 + s1;
      }
    }
    __syncthreads();

    // ---- stream: wavefront w, row group g takes rows w*RPI + g + k*step, U load
    // instructions per batch, the next batch issued before the current is consumed.
    if (on) {
      for (int r = rfirst; r - grp < nb; r += step * U) {
        u32x4 wb[U];
        const bool more = r - grp + step * U < nb;
        if (more) ax_load<T, TL, U>(wb, Mb, rowb, ri, r + step * U, step, nb);
        ax_consume<T, E, U>(wa, cf, r, step, nb, acc);
        if (more) {
#pragma unroll
          for (int u = 0; u < U; ++u) wa[u] = wb[u];
        }
      }
    }
    __syncthreads();
  }
  // ---- combine row groups (lanes with equal lane % TL), then wavefronts, in order
#pragma unroll
  for (int o = TL; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += __shfl_xor(acc[e], o, kWave);
  if (grp == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) red[wave * TL * E + lane * E + e] = acc[e];
  }
  __syncthreads();
  if (tid < TL * E) {
    const int col = blockIdx.x * TL * E + tid;
    if (col < a.d) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w * TL * E + tid];
      if (a.resid) s += a.resid[col];
      if (a.bias) s += a.bias[col];
      a.out[col] = s;
      if (a.out2) a.out2[col] = s;
    }
  }
}

template <typename T, bool HEADS>
static hipError_t launch_axpy_t(AxpyArgs a, hipStream_t st) {
  constexpr int E = Chunk<T>::E;
  const int nch = a.d / E;
  const int tiles = (nch + kAxTL - 1) / kAxTL;
  // LDS budget: 40 KB of (coefficient, row index) pairs plus the combine factors of
  // the heads a batch touches.
  int rpb = 5120;
  size_t fac = 0;
  if (HEADS) {
    for (;;) {
      fac = (size_t)(rpb / a.dh + 2) * a.n_split * 4;
      if (fac <= 16384 || rpb <= 256) break;
      rpb /= 2;
    }
  }
  a.rows_per_batch = max(1, min(rpb, max(a.nrows, 1)));
  size_t lds = (size_t)a.rows_per_batch * 8 + (size_t)kAxNW * kAxTL * E * 4 + fac + 16;
  const int blocks = tiles;
  hipLaunchKernelGGL((k_axpy<T, kAxNW, kAxTL, kAxU, HEADS>), dim3(blocks), dim3(kAxNW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_axpy(int wtype, const AxpyArgs& a, hipStream_t st) {
  if (a.dh > 0)
    return wtype == DV_F16 ? launch_axpy_t<_Float16, true>(a, st) : launch_axpy_t<float, true>(a, st);
  return wtype == DV_F16 ? launch_axpy_t<_Float16, false>(a, st) : launch_axpy_t<float, false>(a, st);
}

}  // namespace dv
