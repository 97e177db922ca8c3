// dv_sparse_block_noalloc: dv_sparse_block with its scratch space in a fixed device
// array of this library instead of a caller workspace, for callers that cannot
// allocate device memory (code being captured into a graph, serving loops that must
// not call the allocator).
//
// `scratch` is a file-scope device array: every device the library runs on holds its
// own copy until the process ends. In host code its name is only a stand-in for the
// symbol, so its device address is looked up once per device (with that device
// current, on the first call there) and that address is what the kernels receive.
// All calls on one device share the array: calls that overlap in time on one device
// race and must be ordered (one stream, or events). Nothing in it has to start at
// zero: the layer's split-sum arrival counters are cleared by an earlier launch of the
// same call, and everything else is written before it is read.
#include <mutex>

#include "dv_internal.hpp"

namespace dv {

static __device__ __align__(256) unsigned char scratch[DV_STATIC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];
}  // namespace

// Device address of this device's copy of `scratch`.
static hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_once[dev], [dev] {
    void* p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_ptr[dev] = p;
  });
  if (g_err[dev] != hipSuccess) return g_err[dev];
  if (g_ptr[dev] == nullptr || (reinterpret_cast<uintptr_t>(g_ptr[dev]) & 255u) != 0) return hipErrorInvalidSymbol;
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace dv

using namespace dv;

extern "C" dv_status dv_sparse_block_noalloc(const dv_attn* a, const dv_mlp* m, const dv_predictor* pa,
                                             const dv_predictor* pm, const dv_ln* ln, const dv_kv* kv,
                                             const float* x_in, float* x_out, int32_t B, int32_t k_heads,
                                             int32_t k_mlp, int32_t mode, int32_t batch_mode, float scale,
                                             int32_t* heads_out, int32_t* idx_out, uint32_t flags, void* stream) {
  // (invalid arguments give 0 here; dv_sparse_block reports them below)
  const size_t need = dv_sparse_block_workspace_bytes(a, m, pa, pm, kv, B, k_heads, k_mlp);
  if (need > (size_t)DV_STATIC_SCRATCH_BYTES) return DV_ERR_WORKSPACE;
  void* ws = nullptr;
  if (scratch_address(&ws) != hipSuccess) return DV_ERR_HIP;
  return dv_sparse_block(a, m, pa, pm, ln, kv, x_in, x_out, B, k_heads, k_mlp, mode, batch_mode, scale, heads_out,
                         idx_out, ws, (size_t)DV_STATIC_SCRATCH_BYTES, flags, stream);
}
