// Device memory of the no-allocation entry point (score_candidates_static): a
// file-scope array that each GPU the library runs on holds from the module's
// load until the process ends. Host code never passes the array's name to a
// kernel or a copy: on the host that name is only a stand-in for the symbol.
// Its device address is looked up once per device with hipGetSymbolAddress,
// with that device current, and that address is what the launches use.
#include <mutex>

#include "tx_internal.h"

namespace tx {

static __device__ __align__(256) char scratch[kStaticScratchBytes];

hipError_t static_scratch(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr_of_device[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr_of_device[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255)) return hipErrorInvalidSymbol;
    addr_of_device[dev] = p;
  }
  *out = addr_of_device[dev];
  return hipSuccess;
}

}  // namespace tx
