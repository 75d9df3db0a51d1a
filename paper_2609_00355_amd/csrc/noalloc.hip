// Static scratch for the entry points that allocate nothing.
//
// A file-scope device array of a fixed size, one copy per GPU, held until the
// process ends.  Host code never passes the array's name to a kernel or a
// copy (in host code it names a host-side stand-in): the device address of
// each GPU's copy is looked up once per device, with that device current, by
// hipGetSymbolAddress, and that address is what the kernels receive.  All
// calls on one GPU share its copy, so calls that overlap on one GPU race.
#include <mutex>

#include "glance_internal.h"

namespace glance {

constexpr size_t kNoAllocScratchBytes = size_t(1) << 20;  // 1 MiB per GPU
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
void* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];
std::once_flag g_once[kMaxDevices];
}  // namespace

size_t noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_once[dev], [dev] {
    void* ptr = nullptr;
    g_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));  // the current device's copy
    g_ptr[dev] = g_err[dev] == hipSuccess ? ptr : nullptr;
  });
  if (g_err[dev] != hipSuccess) return g_err[dev];
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace glance
