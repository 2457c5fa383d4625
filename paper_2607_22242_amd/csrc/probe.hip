// probe.hip -- diagnostics beside the method: the integer VALU throughput
// probe (the empirical ceiling that the search kernel's roofline is read
// against) and a check of the wave-wide OR the search's skipping relies on.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
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

// Lane g takes part when active[g] is non-zero (a divergent branch, as in the
// event loop) and writes the OR over its wave's active lanes of in[g] (64-bit
// form) and of bits 16..47 of in[g] (32-bit form); other lanes write all ones.
__global__ __launch_bounds__(256) void wave_or_probe_kernel(const uint64_t* __restrict__ in,
                                                            const uint8_t* __restrict__ active,
                                                            uint64_t* __restrict__ out64,
                                                            uint32_t* __restrict__ out32) {
  __shared__ uint64_t s_slot[256 / 64];
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  uint64_t* const slot = &s_slot[threadIdx.x / 64];
  uint64_t r64 = ~0ull;
  uint32_t r32 = ~0u;
  if (active[g] != 0) {
    const uint64_t x = in[g];
    r64 = wave_or<uint64_t>(x, slot);
    r32 = wave_or<uint32_t>(uint32_t(x >> 16), reinterpret_cast<uint32_t*>(slot));
  }
  out64[g] = r64;
  out32[g] = r32;
}

hipError_t launch_wave_or_probe(const uint64_t* in, const uint8_t* active, uint32_t blocks,
                                uint64_t* out64, uint32_t* out32, hipStream_t s) {
  hipLaunchKernelGGL(wave_or_probe_kernel, dim3(blocks), dim3(256), 0, s, in, active, out64, out32);
  return hipGetLastError();
}

}  // namespace devmap
