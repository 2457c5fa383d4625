// reduce.h -- lexicographic (makespan, index) minimum across a block, shared
// by the search kernels and the per-table reduction (internal).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "devtab.h"

namespace devmap {

__device__ __forceinline__ void lex_min(uint32_t& ms, uint64_t& x, uint32_t oms, uint64_t ox) {
  if (oms < ms || (oms == ms && ox < x)) {
    ms = oms;
    x = ox;
  }
}

// Block-wide lexicographic min of (makespan, index); result valid in thread 0.
__device__ __forceinline__ void block_min(uint32_t& ms, uint64_t& x) {
  __shared__ uint32_t s_ms[kBlock / 64];
  __shared__ uint64_t s_x[kBlock / 64];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t oms = __shfl_xor(ms, off);
    const uint64_t ox = __shfl_xor(x, off);
    lex_min(ms, x, oms, ox);
  }
  const int wave = threadIdx.x / 64;
  if ((threadIdx.x & 63) == 0) {
    s_ms[wave] = ms;
    s_x[wave] = x;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kBlock / 64; ++w) lex_min(ms, x, s_ms[w], s_x[w]);
  }
}

}  // namespace devmap
