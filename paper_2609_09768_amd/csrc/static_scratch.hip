// Fixed device scratch for the entry point that allocates nothing
// (kvc_blend_prefill_layer_noalloc): a file-scope device array, one copy on
// every GPU the library runs on, held until the process ends.
//
// The array's name is a host-side stand-in on the host: a kernel given it
// would fault.  Host code uses only the address hipGetSymbolAddress returns
// for the current device, looked up once per device and kept here.
#include "kvc_internal.h"

#include <mutex>

static __device__ __align__(256) unsigned char scratch[kvc::kStaticScratchBytes];

namespace kvc {
namespace {

constexpr int kMaxDevices = 256;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices];  // per device ordinal; NULL until looked up

}  // namespace

hipError_t static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace kvc
