// Per-device scratch array of the no-allocation forward entry point.
//
// dtst_forward_noalloc runs the kernels of dtst_forward with this array as
// their workspace, so the call allocates nothing.  The array is a file-scope
// device variable: every GPU the library runs on holds its own copy, at its
// own address, from the time the code object is loaded until the process
// ends.  Host code never uses the array's name as a device address (in host
// code it names a host-side stand-in); the device address is looked up once
// per device with hipGetSymbolAddress, with that device current, and kept.
#include <hip/hip_runtime.h>

#include <mutex>
#include <unordered_map>

#include "dtst_internal.h"

namespace dtst {
namespace {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::unordered_map<int, void*>& scratch_table() {
  static std::unordered_map<int, void*> t;
  return t;
}

}  // namespace

int scratch_address(int device, void** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto& t = scratch_table();
  auto it = t.find(device);
  if (it != t.end()) {
    *out = it->second;
    return hipSuccess;
  }
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) {
    (void)hipGetLastError();  // leave no error behind for the next launch check
    return e;
  }
  if (ptr == nullptr) return hipErrorInvalidSymbol;
  t.emplace(device, ptr);
  *out = ptr;
  return hipSuccess;
}

}  // namespace dtst
