// The workspace of muon_step_static: a fixed-size device array that the
// library itself holds on every GPU it runs on, for callers that cannot
// allocate device memory (code under HIP graph capture, allocation-free
// serving loops).
//
// In host code the array's name is only a stand-in for the symbol, not a
// device address: the address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept in a per-device
// table; only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "muon_internal.h"

namespace {

__device__ __align__(256) char scratch[muon::kStaticWorkspaceBytes];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices] = {};

}  // namespace

namespace muon {

int static_workspace_init(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(g_lock);
  if (!g_scratch[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch[device] = ptr;
  }
  *out = g_scratch[device];
  return hipSuccess;
}

}  // namespace muon
