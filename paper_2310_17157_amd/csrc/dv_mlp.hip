// First half of the sparsified MLP of Eq. (1): for each selected neuron i,
// z_i = x-hat . W^1_i + b1_i and a_i = ReLU(z_i). W^1_i is row i of W1T, so each
// selected neuron is one contiguous row streamed once (Section 4.4 "Kernel fusion":
// the gather is the load itself; nothing is copied). The second half (the a_i-weighted
// sum of rows of W2T) is the gathered row-axpy kernel.
#include "dv_internal.hpp"

namespace dv {

template <typename T, int NW, int S, int U>
__global__ void __launch_bounds__(NW * 64) k_fc1(Fc1Args a) {
  extern __shared__ float smem[];
  constexpr int NT = NW * 64;
  float* xs = smem;
  float* red = smem + a.d;
  float* seg = red + NW;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  constexpr int RPI = NW / S;
  // Issue the first row's loads before the layer-norm prologue.
  u32x4 pf[U];
  {
    const int s0 = blockIdx.x * RPI + wave / S;
    if (s0 < a.k)
      row_prefetch<T, U, S>(static_cast<const T*>(a.W1T) + (size_t)min(max(a.set[s0], 0), a.n - 1) * a.d,
                            a.d, lane, wave % S, pf);
  }
  stage_x<T, NT>(a.x, a.d, a.g, a.be, a.eps, xs, red);
  bool first = true;
  for (int base = blockIdx.x * RPI; base < a.k; base += gridDim.x * RPI) {
    const int s = base + wave / S;
    float v = 0.f;
    int i = 0;
    if (s < a.k) {
      i = min(max(a.set[s], 0), a.n - 1);
      const T* rp = static_cast<const T*>(a.W1T) + (size_t)i * a.d;
      v = first ? wave_rowdot_pf<T, U, S>(rp, xs, a.d, lane, wave % S, pf)
                : wave_rowdot<T, U, S>(rp, xs, a.d, lane, wave % S);
    }
    first = false;
    if constexpr (S > 1) {
      if (lane == 0) seg[wave] = v;
      __syncthreads();
      if (wave % S == 0) {
        float t = 0.f;
#pragma unroll
        for (int j = 0; j < S; ++j) t += seg[wave + j];
        v = t;
      }
      __syncthreads();
    }
    if (wave % S == 0 && lane == 0 && s < a.k) {
      if (a.b1) v += a.b1[i];
      a.h[s] = v > 0.f ? v : 0.f;
    }
  }
}

hipError_t launch_fc1(int wtype, const Fc1Args& a, hipStream_t st) {
  constexpr int NW = 8, S = 2, U = 6;
  constexpr int RPI = NW / S;
  const int blocks = max(1, (a.k + RPI - 1) / RPI);
  const size_t lds = (size_t)(a.d + 2 * NW) * sizeof(float);
  if (wtype == DV_F16)
    hipLaunchKernelGGL((k_fc1<_Float16, NW, S, U>), dim3(blocks), dim3(NW * 64), lds, st, a);
  else
    hipLaunchKernelGGL((k_fc1<float, NW, S, U>), dim3(blocks), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

}  // namespace dv
