// First half of the sparsified MLP of Eq. (1): for each selected neuron i,
// z_i = x-hat . W^1_i + b1_i and a_i = ReLU(z_i). W^1_i is row i of W1T, so each
// selected neuron is one contiguous row streamed once (Section 4.4 "Kernel fusion":
// the gather is the load itself; nothing is copied). One workgroup per CU; rows are
// dealt round-robin over the workgroups (one wavefront per row), so the ~10 rows per
// CU at the OPT-175B shape are balanced to within one. The second half (the
// a_i-weighted sum of rows of W2T) is the gathered row-axpy kernel.
#include "dv_internal.hpp"
#include "dv_rowdot.hpp"

namespace dv {

template <typename T, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_fc1(Fc1Args a) {
  extern __shared__ float smem[];
  float* xs = smem;
  float* red = smem + a.d;
  auto row_ptr = [&](int s) {
    return static_cast<const T*>(a.W1T) + (size_t)min(max(a.set[s], 0), a.n - 1) * a.d;
  };
  auto epi = [&](int s, float v) {
    const int i = min(max(a.set[s], 0), a.n - 1);
    if (a.b1) v += a.b1[i];
    a.h[s] = v > 0.f ? v : 0.f;
  };
  rowdot_wave_loop<T, NW, U>(row_ptr, epi, a.k, a.d, a.x, a.g, a.be, a.eps, xs, red, nullptr, blockIdx.x,
                             gridDim.x);
}

hipError_t launch_fc1(int wtype, const Fc1Args& a, hipStream_t st) {
  constexpr int NW = 16, U = 8;
  const int blocks = max(1, min(a.k, device_cu_count()));
  const size_t lds = (size_t)(a.d + NW) * sizeof(float);
  if (wtype == DV_F16)
    hipLaunchKernelGGL((k_fc1<_Float16, NW, U>), dim3(blocks), dim3(NW * 64), lds, st, a);
  else
    hipLaunchKernelGGL((k_fc1<float, NW, U>), dim3(blocks), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

}  // namespace dv
