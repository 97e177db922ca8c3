// Row-dot loops shared by the predictor's first layer, fc1 and the gathered QKV:
// every selected row (d weights, 16-byte chunks) is dotted with an input vector
// staged once per workgroup in LDS (optionally layer-normalised there).
//
// rowdot_wg_loop: a persistent grid strides over the rows; for each row the NW
// wavefronts of a workgroup split its 16-byte chunks (WgRow), the next row's loads
// are issued before the current row is reduced, and the first row's loads are issued
// before the layer-norm prologue so that HBM latency overlaps it. One barrier per
// row; the per-wavefront partial sums use two alternating LDS slots.
#pragma once

#include "dv_internal.hpp"

namespace dv {

// xs: d floats of LDS; red: NW + 2*NW floats of LDS. row_ptr(row) -> const T*;
// epi(row, value) runs on thread 0. xhat_out (optional) receives the normalised
// input from workgroup 0.
template <typename T, int NW, int JMAX, class RowPtr, class Epi>
__device__ __forceinline__ void rowdot_wg_loop(RowPtr row_ptr, Epi epi, int nrows, int d, const float* x,
                                               const float* g, const float* be, float eps, float* xs,
                                               float* red, float* xhat_out) {
  constexpr int NT = NW * 64;
  constexpr int E = Chunk<T>::E;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = d / E;
  int row = blockIdx.x;
  WgRow<T, NW, JMAX> cur, nxt;
  if (row < nrows) cur.load(row_ptr(row), nch, lane, wave);
  stage_x<T, NT>(x, d, g, be, eps, xs, red);
  if (xhat_out != nullptr && blockIdx.x == 0)
    for (int e = threadIdx.x; e < d; e += NT) xhat_out[e] = xs[xs_index<T>(e, d)];
  float* slots = red + NW;
  int it = 0;
  for (; row < nrows; row += gridDim.x, ++it) {
    const int next = row + gridDim.x;
    if (next < nrows) nxt.load(row_ptr(next), nch, lane, wave);
    const float p = cur.dot(xs, d, nch, lane, wave);
    float* slot = slots + (it & 1) * NW;
    if (lane == 0) slot[wave] = p;
    __syncthreads();
    if (threadIdx.x == 0) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += slot[w];
      epi(row, v);
    }
    cur = nxt;
  }
}

// Wavefront-per-row variant: G workgroups (this is number wg) of NW wavefronts; row r
// goes to workgroup r % G, wavefront (r / G) % NW, so consecutive rows land on different CUs
// and any row count spreads over the machine to within one row per CU. Each
// wavefront streams a whole row with U chunks per lane in flight; its first row's
// loads are issued before the prologue. epi(row, value) runs on lane 0.
template <typename T, int NW, int U, class RowPtr, class Epi>
__device__ __forceinline__ void rowdot_wave_loop(RowPtr row_ptr, Epi epi, int nrows, int d, const float* x,
                                                 const float* g, const float* be, float eps, float* xs,
                                                 float* red, float* xhat_out, int wg, int G) {
  constexpr int NT = NW * 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int row = wg + G * wave;
  u32x4 pf[U];
  if (row < nrows) row_prefetch<T, U, 1>(row_ptr(row), d, lane, 0, pf);
  stage_x<T, NT>(x, d, g, be, eps, xs, red);
  if (xhat_out != nullptr && wg == 0)
    for (int e = threadIdx.x; e < d; e += NT) xhat_out[e] = xs[xs_index<T>(e, d)];
  bool first = true;
  for (; row < nrows; row += G * NW) {
    const T* rp = row_ptr(row);
    const float v = first ? wave_rowdot_pf<T, U, 1>(rp, xs, d, lane, 0, pf) : wave_rowdot<T, U, 1>(rp, xs, d, lane, 0);
    first = false;
    if (lane == 0) epi(row, v);
  }
}

// Chunks per lane needed for a row of nch chunks with NW wavefronts.
inline int rowdot_jmax(int nch, int nw) {
  const int j = (nch + 64 * nw - 1) / (64 * nw);
  return j <= 1 ? 1 : (j <= 2 ? 2 : (j <= 4 ? 4 : 8));
}

}  // namespace dv
