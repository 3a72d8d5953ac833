// scratch.hip -- the library's static device scratch, for callers that cannot allocate.
//
// A file-scope device array that bana_decode_attn_partial_noalloc uses in place of a
// caller workspace (chunk or piece partials and the balanced launch's prefix sums).  Each
// device the library runs on holds its own copy from the time the library's code object
// is loaded there until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up once per device, with
// that device current, and only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

static __device__ __align__(256) unsigned char scratch[bana::kStaticScratchBytes];

namespace bana {
namespace {

constexpr int kMaxDevices = 1024;

std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices];  // device address of `scratch` on each device, once looked up

}  // namespace

hipError_t static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = p;
  }
  *ptr = g_scratch_addr[dev];
  return hipSuccess;
}

}  // namespace bana
