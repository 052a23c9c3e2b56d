// Work-queue counters of the persistent kernels (forward, dK/dV, dQ) and the
// grid of their launches.  The counters of all streams live in one static
// device array per GPU (zero when the code object loads), so handing them out
// allocates nothing and needs no memset: each launch's last workgroup leaves
// its counters at zero again.  Each stream gets its own block, so launches
// that overlap on different streams never share counters; launches on one
// stream are ordered and reuse theirs.  In host code `wq_counters` is only a
// handle: its device address comes from hipGetSymbolAddress, once per device
// with that device current.

#include <hip/hip_runtime.h>

#include <cstdlib>
#include <map>
#include <utility>

#include "zl_internal.h"

namespace {

__device__ __align__(256) int wq_counters[zl::kWqSlots * zl::kWqInts];

constexpr int kMaxDevices = 64;

struct DeviceState {
  int* base = nullptr;                       // device address of this GPU's wq_counters
  std::map<hipStream_t, int> slot_of;        // stream -> block index
  int cus = 0;                               // compute units
  std::map<const void*, int> per_cu;         // kernel -> resident workgroups per CU
};
DeviceState g_dev[kMaxDevices];

bool static_dispatch() {
  static const bool v = [] {
    const char* e = std::getenv("ZL_STATIC_DISPATCH");
    return e && e[0] == '1';
  }();
  return v;
}

}  // namespace

namespace zl {

zl_status stream_counters(hipStream_t s, int** out) {
  *out = nullptr;
  if (static_dispatch()) return ZL_OK;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return host_status(ZL_ERR_HIP, "hipGetDevice failed: no usable GPU");
  if (dev < 0 || dev >= kMaxDevices) return ZL_OK;  // one item per workgroup
  DeviceState& d = g_dev[dev];
  if (!d.base) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(wq_counters)) != hipSuccess || !ptr)
      return host_status(ZL_ERR_HIP, "hipGetSymbolAddress of the work-queue counters failed");
    d.base = static_cast<int*>(ptr);
  }
  auto it = d.slot_of.find(s);
  if (it == d.slot_of.end()) {
    if ((int)d.slot_of.size() >= kWqSlots) return ZL_OK;  // all blocks taken: one item per workgroup
    it = d.slot_of.emplace(s, (int)d.slot_of.size()).first;
  }
  *out = d.base + (size_t)it->second * kWqInts;
  return ZL_OK;
}

int launch_grid(const void* kernel, int block, int n_items, const int* ctr) {
  if (!ctr) return n_items;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return -1;
  DeviceState& d = g_dev[dev];
  if (d.cus == 0 && hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  auto it = d.per_cu.find(kernel);
  if (it == d.per_cu.end()) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, block, 0) != hipSuccess || nb < 1) return -1;
    it = d.per_cu.emplace(kernel, nb).first;
  }
  const long long resident = (long long)it->second * d.cus;
  return (int)(resident < n_items ? resident : n_items);
}

}  // namespace zl
