// The fixed device memory of pat_reducescatter_noalloc.
//
// The entry point that allocates nothing keeps every table, intermediate
// buffer and accumulator its kernels need in `scratch`, a file-scope device
// array of PAT_NOALLOC_SCRATCH_BYTES.  The runtime gives each GPU its own copy
// when it loads this code object; it stays until the process ends.
//
// In host code the array's name stands for a host-side shadow, not for device
// memory: its device address on a GPU comes from hipGetSymbolAddress, taken
// once per device with that device current and kept here, and only that
// address is ever handed to kernels or copies.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/pat.h"
#include "kernels.hpp"

static __device__ __align__(256) unsigned char scratch[PAT_NOALLOC_SCRATCH_BYTES];

namespace pat {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

size_t scratch_bytes() { return sizeof(scratch); }

hipError_t scratch_base(int device, char** base) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    // The caller has made `device` current.
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = static_cast<char*>(ptr);
  }
  *base = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace pat
