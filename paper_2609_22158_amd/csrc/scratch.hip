// Static device scratch for the entry point that allocates nothing
// (stepkv_score_noalloc). The buffer is a file-scope device array: each GPU
// the library runs on holds its own copy until the process ends. In host code
// the array's name is not a device address, so its address on the current
// device is looked up once per device with hipGetSymbolAddress and only that
// pointer is handed to kernels.
#include <mutex>

#include "internal.h"

static __device__ __align__(256) uint8_t scratch[stepkv::kStaticScratchBytes];

namespace stepkv {
namespace {

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];

}  // namespace

hipError_t static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  // once per device, with that device current (the calling thread's)
  std::call_once(g_once[dev], [dev] {
    void* p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_ptr[dev] = g_err[dev] == hipSuccess ? p : nullptr;
  });
  *ptr = g_ptr[dev];
  return g_err[dev];
}

}  // namespace stepkv
