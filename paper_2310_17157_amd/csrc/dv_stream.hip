// A plain streaming read of one contiguous buffer: the measured ceiling that the
// gathered kernels are compared against (the same 16-byte non-temporal loads, with
// no gather, no dependency and no epilogue). Every wavefront reads one contiguous
// share of the buffer, 64 lanes x 16 bytes (1 KB) per load instruction, with two
// batches of U loads in flight, and keeps a running sum of the words it read; a
// wavefront stores its sum only if it equals a value no sum of finite data takes, so
// the loads cannot be dropped and nothing is written in practice. Of the shapes
// measured on this part (grid-stride reads with 4 or 8 loads per thread and 8
// workgroups per CU; contiguous shares with 8 or 16 wavefronts per workgroup, 2-8
// loads per batch, 1 or 2 workgroups per CU), this one is the fastest from 100 MB up
// (557 MB in 84.5 us against 101.8 us for the grid-stride form).
#include "dv_internal.hpp"

namespace dv {

template <int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_stream_read(const u32x4* __restrict__ p, size_t n16, float* sink) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t nwaves = (size_t)gridDim.x * NW, gw = (size_t)blockIdx.x * NW + wave;
  const size_t nslot = n16 / 64;                                 // whole 1 KB slots
  const size_t s0 = gw * nslot / nwaves, s1 = (gw + 1) * nslot / nwaves;
  uint32_t acc = 0u;
  if (s1 > s0) {
    // loads past the share are clamped to its last slot and not used
    auto load = [&](u32x4* w, size_t sb) {
#pragma unroll
      for (int u = 0; u < U; ++u) w[u] = __builtin_nontemporal_load(p + min(sb + u, s1 - 1) * 64 + lane);
    };
    auto use = [&](const u32x4* w, size_t sb) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (sb + u < s1) acc += w[u][0] ^ w[u][1] ^ w[u][2] ^ w[u][3];
    };
    u32x4 wa[U], wb[U];
    load(wa, s0);
    for (size_t sb = s0;;) {
      load(wb, sb + U);
      use(wa, sb);
      sb += U;
      if (sb >= s1) break;
      load(wa, sb + U);
      use(wb, sb);
      sb += U;
      if (sb >= s1) break;
    }
  }
  // the chunks after the last whole slot (fewer than 64): the first wavefront's lanes
  if (gw == 0 && lane < (int)(n16 - nslot * 64)) {
    const u32x4 w = __builtin_nontemporal_load(p + nslot * 64 + lane);
    acc += w[0] ^ w[1] ^ w[2] ^ w[3];
  }
  if (acc == 0x7fc00001u) sink[0] = __uint_as_float(acc);
}

static hipError_t launch_stream_read(const void* buf, size_t n16, float* sink, hipStream_t st) {
  // two workgroups of 16 wavefronts per CU, at most one wavefront per 1 KB slot
  constexpr int NW = 16;
  const size_t want = (size_t)device_cu_count() * 2, need = (n16 / 64 + NW - 1) / NW;
  const int blocks = (int)(want < need ? want : (need > 0 ? need : 1));
  launch_k((k_stream_read<NW, 4>), dim3(blocks), dim3(NW * 64), 0, st, reinterpret_cast<const u32x4*>(buf),
                     n16, sink);
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
