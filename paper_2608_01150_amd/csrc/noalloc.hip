// The allocation-free backward entry point, zl_attn_bwd_noalloc: its work
// tables and its workspace live in a static device array instead of memory
// the library or the caller allocates.  The array is a file-scope device
// variable, so each GPU the library runs on holds its own copy, at its own
// address, from the code object's load until the process ends.  In host code
// the name `scratch` is only a host-side handle: its device address comes from
// hipGetSymbolAddress, looked up once per device with that device current.

#include <hip/hip_runtime.h>

#include <mutex>

#include "zl_attn.h"
#include "zl_internal.h"

namespace {

static __device__ __align__(256) char scratch[ZL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of each GPU's copy of `scratch`

zl_status current_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return zl::host_status(ZL_ERR_HIP, "hipGetDevice failed: no usable GPU");
  if (dev < 0 || dev >= kMaxDevices)
    return zl::host_status(ZL_ERR_UNSUPPORTED, "device index beyond the 64 the scratch table tracks");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return zl::host_status(ZL_ERR_HIP, "hipGetSymbolAddress of the static scratch array failed");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return ZL_OK;
}

}  // namespace

extern "C" zl_status zl_attn_bwd_noalloc(const zl_seg_desc* desc, int32_t num_heads, int32_t head_dim,
                                         zl_dtype dtype, float softmax_scale, const void* q, const void* k,
                                         const void* v, const void* out, const float* lse, const void* dout,
                                         void* dq, void* dk, void* dv, void* stream) {
  return zl::attn_bwd_scratch(desc, num_heads, head_dim, dtype, softmax_scale, q, k, v, out, lse, dout, dq, dk, dv,
                              ZL_NOALLOC_SCRATCH_BYTES, current_scratch, stream);
}
