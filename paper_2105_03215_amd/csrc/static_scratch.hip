// The library's static device scratch: one file-scope array per GPU that
// byoc_subgraph_run_static uses as the intermediate arena of an engine, so
// that run needs no allocation of its own (callers under graph capture or in
// loops that must not call hipMalloc).
//
// The array's name is a host-side stand-in in host code; its device address
// is taken once per device with hipGetSymbolAddress (with that device
// current) and kept in a table.  Host code uses only that address.
#include <hip/hip_runtime.h>

#include <mutex>

#include "static_scratch.h"

namespace byoc {
namespace {

// Held by every GPU the library runs on until the process ends.  `used`
// keeps the otherwise unreferenced array in the code object.
static __device__ __align__(256) __attribute__((used)) char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch_ptr(int device, void** ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[device]) {
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e != hipSuccess) return e;
    if (prev != device && (e = hipSetDevice(device)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev != device) (void)hipSetDevice(prev);
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  return hipSuccess;
}

}  // namespace byoc
