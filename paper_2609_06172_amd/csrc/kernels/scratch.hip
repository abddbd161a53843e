// The library's static device scratch: the workspace of kernels run through
// auvm_run_noalloc (callers that cannot allocate device memory).  The array
// is part of the code object, so each GPU the library runs on holds its own
// copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device, never through the
// array's name (a host-side stand-in).
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace auvm {

namespace {

constexpr uint64_t kScratchBytes = uint64_t(8) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

uint64_t scratch_capacity() { return kScratchBytes; }

hipError_t scratch_address(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[device]) {
    // with `device` current: its own copy of the array
    hipError_t e = hipSetDevice(device);
    if (e != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *out = g_ptr[device];
  return hipSuccess;
}

}  // namespace auvm
