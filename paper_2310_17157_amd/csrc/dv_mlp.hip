// First half of the sparsified MLP of Eq. (1): for each selected neuron i,
// z_i = x-hat . W^1_i + b1_i and a_i = ReLU(z_i). W^1_i is row i of W1T, so each
// selected neuron is one contiguous row streamed once (Section 4.4 "Kernel fusion":
// the gather is the load itself; nothing is copied). One workgroup per CU takes a
// contiguous range of the selected rows and its wavefronts split the range's loads
// evenly (rowdot_flat), so every wavefront of the machine has the same work. The
// second half (the a_i-weighted sum of rows of W2T) is the gathered row-axpy kernel.
#include "dv_internal.hpp"
#include "dv_rowdot.hpp"

namespace dv {

template <typename T, int NW, int U, int KX, bool LN>
__global__ void __launch_bounds__(NW * 64) k_fc1(Fc1Args a) {
  extern __shared__ float smem[];
  float* xs = smem;
  float* red = smem + a.d;
  float* part = red + NW;
  clear_counters(a.clear, a.clear_n);
  auto row_ptr = [&](int s) {
    const size_t row = (size_t)min(max(a.set[s], 0), a.n - 1);
    if constexpr (kIsQ4<T>)
      return static_cast<const char*>(a.W1T) + row * (a.d / 2);
    else
      return static_cast<const T*>(a.W1T) + row * a.d;
  };
  auto scale_ptr = [&](int s) { return a.s1 + (size_t)min(max(a.set[s], 0), a.n - 1) * (a.d / 32); };
  // The epilogue's bias reads: the neuron index of row r0 + tid is read first of all
  // loads (it is not waited for until the end), its bias once the stream is done.
  const int r0 = rowdot_split(blockIdx.x, a.k, gridDim.x), r1 = rowdot_split(blockIdx.x + 1, a.k, gridDim.x);
  const bool mine = (int)threadIdx.x < r1 - r0;
  // (with no rows the set may be NULL: a valid word of the input is read instead)
  const int32_t* sp = a.k > 0 ? a.set + min(r0 + (int)threadIdx.x, a.k - 1) : reinterpret_cast<const int32_t*>(a.x);
  const int sraw = *sp;   // clamped at use
  float bias = 0.f;
  auto tail = [&]() {
    if (mine && a.b1) bias = a.b1[min(max(sraw, 0), a.n - 1)];
  };
  auto epi = [&](int s, float v) {
    if (s - r0 == (int)threadIdx.x) {
      v += bias;
    } else if (a.b1) {
      v += a.b1[min(max(a.set[s], 0), a.n - 1)];
    }
    a.h[s] = act_apply(v, a.act);
  };
  rowdot_flat<T, NW, U, KX, LN>(row_ptr, epi, a.k, a.d, a.x, a.g, a.be, a.eps, xs, red, part, nullptr, blockIdx.x,
                                gridDim.x, tail, scale_ptr);
}

template <typename T, int KX>
static hipError_t launch_fc1_t(const Fc1Args& a, hipStream_t st) {
  // two batches of 2 loads in flight per wavefront: measured faster than all of a
  // wavefront's loads at once (12 at the OPT-175B shape) or batches of 1, 3, 4 or 6,
  // as deeper queues let the XCDs that win the fabric arbitration run ahead
  constexpr int NW = 16, U = 2;
  const int blocks = max(1, min(a.k, device_cu_count()));
  const size_t lds = (size_t)(a.d + NW + rowdot_flat_part(a.k, blocks, NW)) * sizeof(float);
  const void* kern = a.g != nullptr ? reinterpret_cast<const void*>(k_fc1<T, NW, U, KX, true>)
                                    : reinterpret_cast<const void*>(k_fc1<T, NW, U, KX, false>);
  const hipError_t e = ensure_dyn_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (a.g != nullptr)
    launch_k((k_fc1<T, NW, U, KX, true>), dim3(blocks), dim3(NW * 64), lds, st, a);
  else
    launch_k((k_fc1<T, NW, U, KX, false>), dim3(blocks), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_fc1_k(const Fc1Args& a, hipStream_t st) {
  switch (rowdot_kx(a.d, 16)) {
    case 1: return launch_fc1_t<T, 1>(a, st);
    case 2: return launch_fc1_t<T, 2>(a, st);
    case 3: return launch_fc1_t<T, 3>(a, st);
    default: return launch_fc1_t<T, 4>(a, st);
  }
}

hipError_t launch_fc1(int wtype, const Fc1Args& a, hipStream_t st) {
  if (wtype == DV_Q4) return launch_fc1_k<q4_t>(a, st);
  return wtype == DV_F16 ? launch_fc1_k<_Float16>(a, st) : launch_fc1_k<float>(a, st);
}

}  // namespace dv
