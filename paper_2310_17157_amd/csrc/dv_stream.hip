// A plain streaming read of one contiguous buffer: the measured ceiling that the
// gathered kernels are compared against (the same 16-byte non-temporal loads, with
// no gather, no dependency and no epilogue). Each thread reads 16-byte chunks at a
// grid stride, U loads in flight, and keeps a running sum of the words it read; a
// workgroup stores its sum only if it equals a value no sum of finite data takes,
// so the loads cannot be dropped and nothing is written in practice.
#include "dv_internal.hpp"

namespace dv {

template <int U>
__global__ void __launch_bounds__(256) k_stream_read(const u32x4* __restrict__ p, size_t n16, float* sink) {
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    u32x4 w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc += w[u][0] ^ w[u][1] ^ w[u][2] ^ w[u][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 w = __builtin_nontemporal_load(p + i);
    acc += w[0] ^ w[1] ^ w[2] ^ w[3];
  }
  if (acc == 0x7fc00001u) sink[0] = __uint_as_float(acc);
}

static hipError_t launch_stream_read(const void* buf, size_t n16, float* sink, hipStream_t st) {
  // 8 workgroups of 256 threads per CU, 4 loads in flight per thread
  const size_t want = (size_t)device_cu_count() * 8, need = (n16 + 255) / 256;
  const int blocks = (int)(want < need ? want : need);
  hipLaunchKernelGGL(k_stream_read<4>, dim3(blocks), dim3(256), 0, st, reinterpret_cast<const u32x4*>(buf), n16,
                     sink);
  return hipGetLastError();
}

}  // namespace dv

using namespace dv;

extern "C" dv_status dv_stream_read(const void* buf, size_t bytes, float* sink, void* stream) {
  trace_reset();
  if (buf == nullptr || sink == nullptr) return DV_ERR_NULL;
  if (!aligned16(buf) || (bytes & 15u) != 0) return DV_ERR_ALIGN;
  if (bytes == 0) return DV_OK;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  DV_LAUNCH("stream_read", hs, launch_stream_read(buf, bytes / 16, sink, hs));
  return DV_OK;
}
