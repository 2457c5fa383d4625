// scratch.hip -- the device memory of the entry point that allocates nothing
// (sched_bruteforce_argmin_noalloc): one fixed array per GPU, holding what a
// caller-provided workspace holds otherwise (problem table, per-block
// partial minima, result).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "launch.h"

namespace devmap {

// Each GPU the library runs on holds its own copy until the process ends.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_ptr[kMaxDevices];  // device address of scratch on each GPU, once looked up

}  // namespace

// Device address of the calling thread's current GPU's scratch array.  The
// array's host-side name is not a device address: the address is looked up
// once per device with hipGetSymbolAddress (with that device current) and
// kept.
hipError_t scratch_buffer(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace devmap
