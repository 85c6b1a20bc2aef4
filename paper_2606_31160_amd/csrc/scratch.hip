// The library's static per-device scratch array, used by spec_verify_scratch
// for the per-pass partial results, arrival counters and logits staging that
// spec_verify keeps in the context's workspace.
//
// The array is part of the code object: every GPU the library is loaded on
// holds its own copy, at its own address, until the process ends, and no call
// allocates it.  In host code the array's name only stands for the device
// symbol; its device address is looked up once per device with
// hipGetSymbolAddress (scratch_resolve, called by spec_init with that device
// current) and only that address is handed to kernels and fill launches.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ctx.h"

namespace specdec {

namespace {

static __device__ __align__(256) unsigned char scratch[SPEC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t scratch_resolve(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_ptr[device]) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p) return hipErrorInvalidSymbol;
  g_ptr[device] = p;
  return hipSuccess;
}

void* scratch_device_ptr(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_mu);
  return g_ptr[device];
}

size_t scratch_capacity() { return SPEC_SCRATCH_BYTES; }

}  // namespace specdec
