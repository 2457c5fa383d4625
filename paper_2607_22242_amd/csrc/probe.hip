// probe.hip -- integer VALU throughput probe: the empirical ceiling that the
// search kernel's roofline is read against.  Not part of the method.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace devmap {

constexpr uint32_t kProbeChains = 8;  // independent dependency chains per lane
constexpr uint32_t kProbeOps = 4;     // add, max, compare, select per chain step

__global__ __launch_bounds__(256) void valu_probe_kernel(uint32_t iters, uint32_t seed,
                                                         uint32_t* __restrict__ out) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  const uint32_t x = seed ^ g, y = seed * 3u + g, z = seed + (g << 3), w = g * 0x9E3779B9u;
  uint32_t a[kProbeChains];
#pragma unroll
  for (uint32_t j = 0; j < kProbeChains; ++j) a[j] = g + j * 0x01234567u;
  for (uint32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (uint32_t j = 0; j < kProbeChains; ++j) {
      uint32_t v = a[j] + x;  // add
      v = v > y ? v : y;      // max
      a[j] = v > z ? v : w;   // compare, select
    }
  }
  uint32_t r = 0;
#pragma unroll
  for (uint32_t j = 0; j < kProbeChains; ++j) r ^= a[j];
  out[g] = r;
}

hipError_t launch_valu_probe(uint32_t blocks, uint32_t iters, uint32_t* out, hipStream_t s,
                             double* lane_ops) {
  *lane_ops = double(blocks) * 256.0 * double(iters) * double(kProbeChains * kProbeOps);
  hipLaunchKernelGGL(valu_probe_kernel, dim3(blocks), dim3(256), 0, s, iters, 0x5EEDu, out);
  return hipGetLastError();
}

}  // namespace devmap
