// The library's own scratch memory for the workspace-free layer call
// (mira_moe_forward_noalloc): a file-scope device array that takes the place
// of the caller's workspace, for callers that cannot allocate device memory.
//
// Every device the library runs on holds its own copy of the array until the
// process ends.  In host code the array's name is only a host-side stand-in,
// so its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// ever passed on.  All calls on one device share the array: calls that
// overlap in time on one device race on it.  Nothing in it needs to start at
// zero: the layer's kernels write every workspace region before reading it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "mira_internal.h"

static __device__ __align__(256) unsigned char scratch[MIRA_NOALLOC_SCRATCH_BYTES];

namespace mira {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255)) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace mira
