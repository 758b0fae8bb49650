// Device scratch for the allocation-free decode entry point
// (sfa_attn_decode_noalloc), for callers that cannot allocate device memory
// around a call.
//
// The scratch is a file-scope device array: every GPU the library runs on
// holds its own copy, at its own address, until the process ends.  Host code
// never passes the array's name to a kernel (on the host that name is only a
// stand-in symbol); it looks the device address up once per device with
// hipGetSymbolAddress, with that device current, and uses that address.
//
// Every call on one GPU shares that GPU's copy and leaves its contents
// behind.  The decode writes each partial slot before the merge reads it, so
// nothing in the scratch has to start at zero; calls that overlap in time on
// one GPU race on it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/sfa.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr size_t kScratchBytes = SFA_DECODE_NOALLOC_MAX_BYTES;  // per GPU

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device

}  // namespace

size_t noalloc_scratch_bytes() { return kScratchBytes; }

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace sfa
