// dispatch.hip -- run-time dispatch on the tool count, and the final
// per-table argmin reduction.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <array>
#include <utility>

#include "devtab.h"
#include "launch.h"
#include "reduce.h"

namespace devmap {

template <int N>
hipError_t launch_search_n(const SearchArgs& a, hipStream_t s);
template <int N>
hipError_t launch_eval_n(const uint32_t* tab, const uint64_t* idx, int64_t n, uint64_t n_mappings,
                         int64_t* out, uint32_t sharing, hipStream_t s);
template <int N>
hipError_t launch_bound_n(const uint32_t* tab, uint32_t K, uint64_t known, int64_t n,
                          uint32_t ub, uint32_t* count, uint2* out, hipStream_t s);

// Per-table minimum over its blocks' partials.
__global__ __launch_bounds__(kBlock) void reduce_kernel(const Partial* __restrict__ partials,
                                                        uint32_t per_table,
                                                        DevResult* __restrict__ out) {
  const Partial* p = partials + size_t(blockIdx.x) * per_table;
  uint32_t ms = kInf;
  uint64_t x = ~0ull;
  for (uint32_t i = threadIdx.x; i < per_table; i += kBlock) lex_min(ms, x, p[i].makespan, p[i].index);
  block_min(ms, x);
  if (threadIdx.x == 0) {
    DevResult r;
    r.index = (ms == kInf) ? ~0ull : x;
    r.makespan = (ms == kInf) ? INT64_MAX : int64_t(ms);
    out[blockIdx.x] = r;
  }
}

using SearchFn = hipError_t (*)(const SearchArgs&, hipStream_t);
using EvalFn = hipError_t (*)(const uint32_t*, const uint64_t*, int64_t, uint64_t, int64_t*,
                              uint32_t, hipStream_t);

template <size_t... I>
static constexpr auto make_search_table(std::index_sequence<I...>) {
  return std::array<SearchFn, sizeof...(I)>{&launch_search_n<int(I) + 1>...};
}
template <size_t... I>
static constexpr auto make_eval_table(std::index_sequence<I...>) {
  return std::array<EvalFn, sizeof...(I)>{&launch_eval_n<int(I) + 1>...};
}
using BoundFn = hipError_t (*)(const uint32_t*, uint32_t, uint64_t, int64_t, uint32_t, uint32_t*,
                               uint2*, hipStream_t);
template <size_t... I>
static constexpr auto make_bound_table(std::index_sequence<I...>) {
  return std::array<BoundFn, sizeof...(I)>{&launch_bound_n<int(I) + 1>...};
}

static const auto kSearchFns = make_search_table(std::make_index_sequence<kMaxTools>{});
static const auto kEvalFns = make_eval_table(std::make_index_sequence<kMaxTools>{});
static const auto kBoundFns = make_bound_table(std::make_index_sequence<kMaxTools>{});

hipError_t launch_search(int n_tools, const SearchArgs& a, hipStream_t s) {
  return kSearchFns[n_tools - 1](a, s);
}

hipError_t launch_eval(int n_tools, const uint32_t* tab, const uint64_t* idx, int64_t n,
                       uint64_t n_mappings, int64_t* out, uint32_t sharing, hipStream_t s) {
  return kEvalFns[n_tools - 1](tab, idx, n, n_mappings, out, sharing, s);
}

hipError_t launch_bound(int n_tools, const uint32_t* tab, uint32_t K, uint64_t known, int64_t n,
                        uint32_t ub, uint32_t* count, uint2* out, hipStream_t s) {
  return kBoundFns[n_tools - 1](tab, K, known, n, ub, count, out, s);
}

hipError_t launch_reduce(const Partial* partials, uint32_t per_table, uint32_t n_tables,
                         DevResult* out, hipStream_t s) {
  hipLaunchKernelGGL(reduce_kernel, dim3(n_tables), dim3(kBlock), 0, s, partials, per_table,
                     out);
  return hipGetLastError();
}

}  // namespace devmap
