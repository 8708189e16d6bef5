// Selection workspace held by the library itself, for callers that cannot
// allocate device memory (code under stream capture, tight serving loops,
// harnesses that forbid allocation): a file-scope device array of
// kStaticWorkspaceBytes, one copy per GPU, alive until the process ends.
//
// In host code the array's name is only a host-side handle: the device address
// of each GPU's copy comes from hipGetSymbolAddress, taken once per device
// (with that device current) on the first call there, and that address is what
// the kernels receive.  Every call on a GPU shares its copy, which keeps the
// last call's contents; the selection kernels initialise whatever they read
// (the workspace contract), and calls that overlap on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.h"

namespace vecattn {
namespace {

__device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of each GPU's copy (nullptr: not yet taken)

}  // namespace

hipError_t static_workspace(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

}  // namespace vecattn
