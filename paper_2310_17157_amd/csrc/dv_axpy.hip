// Gathered row-axpy: out = resid + bias + sum_rows coef[row] * M[rowidx(row), :].
//
// This is the second half of both sparsified blocks: the MLP's
// sum_{i in S_M} ReLU(z_i) W^2_i over rows of W2T (Eq. (1)), and the attention's
// sum_{i in S_A} H_i(y) W^O_i over the dh rows of each selected head in WoT (Eq. (2)).
// Both weights are stored transposed so that a selected neuron or head is a set of
// whole contiguous rows (Section 4.4 "Memory coalescing").
//
// Tiling: a workgroup owns one column tile (64 lanes x one 16-byte chunk = 1 KB of
// fp16) and a contiguous range of selected rows; each wavefront streams every NW-th
// row of that range with U rows in flight and accumulates in registers. Wavefront
// partials are summed in LDS in a fixed order and written per row range; a small
// second kernel (k_reduce) adds the ranges in order plus residual and bias. No
// floating-point atomics and no device-scope fences (on a multi-XCD part a
// device-scope release writes back the XCD's L2, which costs far more than a second
// launch): the result is bitwise reproducible.
//
// For the attention, the coefficients H_i(y)[t] are first combined from the split-KV
// partials (max logit, sum of exponentials, unnormalised value sums per chunk).
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

constexpr int kAxpyNW = 8;
constexpr int kAxpyU = 8;

template <typename T, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_axpy(AxpyArgs a) {
  constexpr int E = Chunk<T>::E;
  extern __shared__ float smem[];
  const int tile = blockIdx.x, split = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = a.d / E;
  const int c = tile * 64 + lane;
  const int r0 = split * a.rows_per_split;
  const int nloc = max(0, min(a.nrows, r0 + a.rows_per_split) - r0);
  float* cf = smem;                                        // rows_per_split
  int* ri = reinterpret_cast<int*>(cf + a.rows_per_split); // rows_per_split
  float* red = reinterpret_cast<float*>(ri + a.rows_per_split);   // NW * 64 * E

  for (int i = threadIdx.x; i < nloc; i += NW * 64) {
    const int row = r0 + i;
    if (a.dh == 0) {
      cf[i] = a.coef[row];
      ri[i] = min(max(a.set[row], 0), a.m_rows - 1);
    } else {
      const int j = row / a.dh, t = row - j * a.dh;
      if (a.coef != nullptr) {
        cf[i] = a.coef[row];
      } else {
        const float* P = a.part + (size_t)j * a.n_split * (a.dh + 2);
        float M = -INFINITY;
        for (int s = 0; s < a.n_split; ++s) M = fmaxf(M, P[(size_t)s * (a.dh + 2)]);
        float L = 0.f, O = 0.f;
        for (int s = 0; s < a.n_split; ++s) {
          const float ms = P[(size_t)s * (a.dh + 2)];
          const float f = ms == -INFINITY ? 0.f : __expf(ms - M);
          L += P[(size_t)s * (a.dh + 2) + 1] * f;
          O += P[(size_t)s * (a.dh + 2) + 2 + t] * f;
        }
        cf[i] = O / L;
      }
      ri[i] = min(max(a.set[j], 0), a.m_rows / a.dh - 1) * a.dh + t;
    }
  }
  __syncthreads();

  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  if (c < nch) {
    const char* Mb = static_cast<const char*>(a.M) + (size_t)c * 16;
    const size_t rowb = (size_t)a.d * sizeof(T);
    int i = wave;
    for (; i + NW * (U - 1) < nloc; i += NW * U) {
      u32x4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) w[u] = ld_stream(Mb + (size_t)ri[i + NW * u] * rowb);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float v[E];
        unpack<T>(w[u], v);
        const float f = cf[i + NW * u];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(f, v[e], acc[e]);
      }
    }
    for (; i < nloc; i += NW) {
      u32x4 w = ld_stream(Mb + (size_t)ri[i] * rowb);
      float v[E];
      unpack<T>(w, v);
      const float f = cf[i];
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(f, v[e], acc[e]);
    }
  }
  // Wavefront partials -> LDS -> fixed-order sum by wavefront 0.
#pragma unroll
  for (int e = 0; e < E; ++e) red[(wave * E + e) * 64 + lane] = acc[e];
  __syncthreads();
  const bool single = gridDim.y == 1;
  if (wave == 0 && c < nch) {
    float s[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) t += red[(w * E + e) * 64 + lane];
      s[e] = t;
    }
    if (single) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int col = c * E + e;
        float v = s[e];
        if (a.resid) v += a.resid[col];
        if (a.bias) v += a.bias[col];
        a.out[col] = v;
        if (a.out2) a.out2[col] = v;
      }
    } else {
      float* P = a.partial + (size_t)split * a.d + (size_t)c * E;
#pragma unroll
      for (int e = 0; e < E; ++e) P[e] = s[e];
    }
  }
}

// out[c] = resid[c] + bias[c] + sum_{s < nsplit} partial[s][c]. A workgroup covers 64
// float4 columns with 4 thread groups; group g sums the splits s = g (mod 4) in
// increasing order, then the 4 group sums are added in order g = 0..3: a fixed
// association, so the result is bitwise reproducible.
__global__ void __launch_bounds__(256) k_reduce(const float* __restrict__ partial, int nsplit, int d,
                                                const float* __restrict__ resid, const float* __restrict__ bias,
                                                float* __restrict__ out, float* __restrict__ out2) {
  __shared__ f32x4 part[4][64];
  const int col = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int c4 = blockIdx.x * 64 + col;
  const bool on = c4 * 4 < d;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (on) {
    int sp = g;
    for (; sp + 12 < nsplit; sp += 16) {
      f32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4*>(partial + (size_t)(sp + 4 * u) * d + 4 * c4);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc += v[u];
    }
    for (; sp < nsplit; sp += 4) acc += *reinterpret_cast<const f32x4*>(partial + (size_t)sp * d + 4 * c4);
  }
  part[g][col] = acc;
  __syncthreads();
  if (g == 0 && on) {
    f32x4 t = part[0][col];
    t += part[1][col];
    t += part[2][col];
    t += part[3][col];
    if (resid) t += *reinterpret_cast<const f32x4*>(resid + 4 * c4);
    if (bias) t += *reinterpret_cast<const f32x4*>(bias + 4 * c4);
    *reinterpret_cast<f32x4*>(out + 4 * c4) = t;
    if (out2) *reinterpret_cast<f32x4*>(out2 + 4 * c4) = t;
  }
}

hipError_t launch_reduce(const float* partial, int nsplit, int d, const float* resid, const float* bias,
                         float* out, float* out2, hipStream_t st) {
  const int n4 = d / 4;
  hipLaunchKernelGGL(k_reduce, dim3((n4 + 63) / 64), dim3(256), 0, st, partial, nsplit, d, resid, bias, out,
                     out2);
  return hipGetLastError();
}

int axpy_tiles(int d, int wtype) {
  const int nch = d / (16 / elem_bytes(wtype));
  return (nch + 63) / 64;
}

int axpy_rsplit(int nrows, int d, int wtype, int* rows_per_split) {
  // Aim for about 4 workgroups per CU in total, with at least 4 rows per wavefront
  // where possible and at most 64 row ranges.
  if (nrows <= 0) {
    *rows_per_split = 1;
    return 1;
  }
  const int tiles = axpy_tiles(d, wtype);
  const int target = 4 * device_cu_count();
  int splits = (target + tiles - 1) / tiles;
  const int min_rows = kAxpyNW * 4;
  splits = max(1, min(splits, (nrows + min_rows - 1) / min_rows));
  splits = min(splits, 64);
  int rps = (nrows + splits - 1) / splits;
  splits = (nrows + rps - 1) / rps;
  *rows_per_split = max(rps, 1);
  return max(splits, 1);
}

template <typename T>
static hipError_t launch_axpy_t(const AxpyArgs& a, hipStream_t st) {
  constexpr int NW = kAxpyNW, U = kAxpyU;
  constexpr int E = Chunk<T>::E;
  const int tiles = axpy_tiles(a.d, sizeof(T) == 2 ? DV_F16 : DV_F32);
  const size_t lds = (size_t)a.rows_per_split * 8 + (size_t)NW * 64 * E * sizeof(float);
  hipLaunchKernelGGL((k_axpy<T, NW, U>), dim3(tiles, a.n_rsplit), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_axpy(int wtype, const AxpyArgs& a, hipStream_t st) {
  return wtype == DV_F16 ? launch_axpy_t<_Float16>(a, st) : launch_axpy_t<float>(a, st);
}

}  // namespace dv
