// Fixed device scratch for the entry point that allocates nothing
// (erc_sampling_probs_static): the reduction levels, tickets and totals of the
// sampling-probability kernels live in one file-scope device array instead of a
// caller-provided buffer.  Each GPU holds its own copy of the array, at its own address,
// for the life of the process.  In host code the array's name is only a stand-in for
// that address, so the address is looked up once per device, with that device current,
// and only the looked-up pointer is passed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "erc_common.h"

namespace erc {
namespace {

constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch_setup(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device] != nullptr) return hipSuccess;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != device) return hipErrorInvalidDevice;  // the caller makes the device current
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (p == nullptr) return hipErrorInvalidSymbol;
  g_scratch_ptr[device] = p;
  return hipSuccess;
}

void* static_scratch_ptr(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[device];
}

}  // namespace erc
