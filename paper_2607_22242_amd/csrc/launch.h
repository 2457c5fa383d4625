// launch.h -- host-side entry points into the kernels (internal).
#pragma once
#include <hip/hip_runtime.h>

#include "devtab.h"

namespace devmap {

hipError_t launch_search(int n_tools, const SearchArgs& a, hipStream_t s);
hipError_t launch_eval(int n_tools, const uint32_t* tab, const uint64_t* idx, int64_t n,
                       uint64_t n_mappings, int64_t* out, uint32_t sharing, hipStream_t s);
hipError_t launch_bound(int n_tools, const uint32_t* tab, uint32_t K, uint64_t known, int64_t n,
                        uint32_t ub, uint32_t* count, uint2* out, hipStream_t s);
hipError_t launch_reduce(const Partial* partials, uint32_t per_table, uint32_t n_tables,
                         DevResult* out, hipStream_t s);
// Bytes of the per-GPU scratch array of the entry point that allocates
// nothing: one problem table, 65,536 block partials and a result fit.
constexpr size_t kScratchBytes = size_t(2) << 20;
hipError_t scratch_buffer(void** ptr);
hipError_t launch_wave_or_probe(const uint64_t* in, const uint8_t* active, uint32_t blocks,
                                uint64_t* out64, uint32_t* out32, hipStream_t s);
hipError_t launch_valu_probe(uint32_t blocks, uint32_t iters, uint32_t* out, hipStream_t s,
                             double* lane_ops);

}  // namespace devmap
