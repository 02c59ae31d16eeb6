// Static per-device scratch for the no-allocation forward entry point (fs_slice_fwd_noalloc).
//
// The slice pass needs device memory beyond its inputs and outputs: the per-workgroup
// partial sums of U and s, and for the slot-blocked kernels the per-point normaliser when the
// caller passes no lse buffer. fs_slice_fwd takes it from a caller workspace; the no-allocation
// variant takes it from the file-scope array below, which the code-object loader places in
// every GPU's memory when the library's kernels are first loaded there, and which stays there
// until the process ends. Its host-side name is only a handle for the runtime: the device
// address of each GPU's copy comes from hipGetSymbolAddress with that GPU current, once, and
// only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "fs_internal.h"

namespace fs {
namespace {

__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device] == nullptr) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
  }
  *ptr = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace fs
