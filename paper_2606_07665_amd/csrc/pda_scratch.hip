// Fixed device scratch of the attention entry point that allocates nothing
// (paged_decode_attention_noalloc): the split partials, the steps prefix and
// the split list live in this file-scope array instead of a per-stream
// workspace from hipMalloc.  Each device the library runs on holds its own
// copy until the process ends.
//
// In host code `scratch` names a host-side stand-in, not the device memory:
// the device address comes from hipGetSymbolAddress, taken once per device
// (with that device current) and kept; kernels receive only that address.
#include <hip/hip_runtime.h>

#include <mutex>

#include "pda.h"
#include "pda_internal.h"

namespace pda {

static __device__ __align__(256) unsigned char scratch[PDA_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(int dev, void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace pda
