// Fixed device scratch of jet_score_candidates_noalloc: a file-scope device
// array that every GPU the library runs on holds for the life of the
// process, so that the entry point carves its work buffers from it instead
// of calling hipMalloc.
//
// In host code the array's name is a host-side stand-in, not a device
// address: the address is looked up once per device (hipGetSymbolAddress,
// with that device current) when a model is loaded on it, and only that
// address is ever handed to kernels or copies.
#include <mutex>

#include "noalloc.h"

namespace jet {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {
std::mutex g_mu;
void *g_scratch[kNoallocMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch_init(int device) {
  if (device < 0 || device >= kNoallocMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[device]) return hipSuccess;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != device) return hipErrorInvalidDevice;  // the caller makes the device current
  void *p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p) return hipErrorInvalidSymbol;
  g_scratch[device] = p;
  return hipSuccess;
}

void *noalloc_scratch(int device) {
  if (device < 0 || device >= kNoallocMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  return g_scratch[device];
}

}  // namespace jet
