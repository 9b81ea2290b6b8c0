// Device scratch of the allocation-free run_mutants entry point: one
// file-scope array per GPU, of a fixed size, that holds the chunk activation
// workspace and the per-mutant kill counts and label masks of a call, so the
// call itself never allocates device memory.
//
// In host code the name `scratch` is only a host-side stand-in for the
// array; its device address is looked up once per device (with that device
// current) through hipGetSymbolAddress and kept here, and only that address is
// ever handed to kernels or copies.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/mure.h"
#include "kernels.hpp"

namespace mure {

static __device__ __align__(256) unsigned char scratch[MURE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_mutex;
void* g_ptr[MAX_DEVICES] = {};
}  // namespace

// Device address of this GPU's scratch array (device must be current).
hipError_t noalloc_scratch(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_ptr[device]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *out = g_ptr[device];
  return hipSuccess;
}

}  // namespace mure
