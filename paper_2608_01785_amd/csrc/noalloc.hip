// Library-owned device scratch for callers that cannot allocate device
// memory (tight serving loops, harnesses that forbid allocation): the
// workspace of hs_downstream_decode_step_noalloc lives in one file-scope
// device array instead of a caller buffer.
//
// The array exists once per GPU the library runs on and stays allocated until
// the process ends.  In host code its name is a host-side stand-in, not a
// device address; its address on a device comes from hipGetSymbolAddress
// with that device current, resolved once per device (at context creation)
// and kept here.  Every call on a GPU shares that GPU's array: calls that
// overlap on one GPU race.  The array keeps the last call's contents; what a
// call needs zeroed (its arrival counters) arrives with its metadata copy.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hs_kernels.h"

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

namespace hs {

size_t noalloc_scratch_bytes() { return kScratchBytes; }

hipError_t noalloc_scratch_resolve(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_addr[device] = p;
  }
  *out = g_addr[device];
  return hipSuccess;
}

}  // namespace hs
