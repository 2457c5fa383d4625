// kernels.h -- HIP kernels for gfx950: base-3 mapping decode, integer
// event-driven schedule evaluation, and (makespan, index) argmin reduction.
//
// One lane scores one mapping at a time.  Its per-tool times live in VGPRs
// (the loops over tools are unrolled for a compile-time tool count N), the
// tool constants are wave-uniform scalar loads, and the contention-scaled
// duration table sits in LDS.  A lane owns one "outer" combination (the modes
// of tools J..N-1, decoded once) and walks all 3^J "inner" combinations of
// tools 0..J-1 with a wave-uniform odometer, so the inner modes cost scalar
// instructions only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <array>
#include <type_traits>
#include <utility>

#include "devtab.h"
#include "launch.h"

namespace devmap {

template <int N>
using MaskT = typename std::conditional<(N <= 32), uint32_t, uint64_t>::type;

// A wave-uniform value (scalar register); the identity in a host build.
#if defined(__HIP_DEVICE_COMPILE__)
#define DEVMAP_UNIFORM(x) __builtin_amdgcn_readfirstlane(x)
#else
#define DEVMAP_UNIFORM(x) (x)
#endif

__host__ __device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }
__host__ __device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }

template <int N>
__host__ __device__ __forceinline__ MaskT<N> all_tools() {
  if constexpr (N == 32) return 0xFFFFFFFFu;
  else if constexpr (N == 64) return ~0ull;
  else return (MaskT<N>(1) << N) - 1;
}

template <int N>
__host__ __device__ __forceinline__ MaskT<N> load_mask(const uint32_t* tab, uint32_t lo_word) {
  if constexpr (N <= 32) return tab[lo_word];
  else return uint64_t(tab[lo_word]) | (uint64_t(tab[lo_word + 1]) << 32);
}

template <int N>
__host__ __device__ __forceinline__ bool bit(MaskT<N> m, int v) {
  return (m >> v) & 1;
}

// Makespan of one mapping under the schedule model, or kInf if infeasible.
//
// gnm / gqm: tools on gpu_now / gpu_queue (the rest run on the CPU).
// T[v] holds tool v's ready time while it waits (kInf until all of its
// predecessors have started) and its finish time once it has started.  Each
// pass of the loop handles one event time t:
//   release (implicit: a started GPU tool runs while T > t), immediate starts
//   of cpu / gpu_now tools ready at t with the out-of-memory check, one FIFO
//   queue admission, contention-scaled durations with k counting co-starters,
//   ready times of tools whose predecessors have all started, next event.
template <int N>
__host__ __device__ __forceinline__ uint32_t evaluate(const uint32_t* __restrict__ tab,
                                             const uint32_t* __restrict__ s_dur,
                                             uint32_t levels, uint32_t budget,
                                             MaskT<N> gnm, MaskT<N> gqm) {
  using M = MaskT<N>;
  const M ALL = all_tools<N>();
  const M gpum = gnm | gqm;
  if (gpum & load_mask<N>(tab, kHdrBigLo)) return kInf;  // footprint > budget
  const M src = load_mask<N>(tab, kHdrSrcLo);

  uint32_t T[N];
#pragma unroll
  for (int v = 0; v < N; ++v) T[v] = bit<N>(src, v) ? 0u : kInf;

  M started = 0;
  uint32_t t = 0;
  uint32_t qfin = 0;  // finish time of the running queued tool (0: none)
  uint32_t result = kInf;

  for (int pass = 0; pass < 2 * N + 2; ++pass) {
    // GPU tools still running at t, and the VRAM they hold.
    const M sg = started & gpum;
    uint32_t in_use = 0, k = 0;
#pragma unroll
    for (int v = 0; v < N; ++v) {
      if (bit<N>(sg, v) && T[v] > t) {
        in_use += tab[kHdrWords + kToolWords * v + kToolMem];
        k += 1;
      }
    }
    // Immediate starts: waiting cpu / gpu_now tools whose ready time is t.
    const M cand = ~started & ~gqm & ALL;
    M st = 0;
#pragma unroll
    for (int v = 0; v < N; ++v)
      if (bit<N>(cand, v) && T[v] == t) st |= M(1) << v;
    const M stgn = st & gnm;
#pragma unroll
    for (int v = 0; v < N; ++v) {
      if (bit<N>(stgn, v)) {
        in_use += tab[kHdrWords + kToolWords * v + kToolMem];
        k += 1;
      }
    }
    if (in_use > budget) break;  // out of memory: infeasible

    // Serialized queue: admit the ready queued tool with the smallest
    // (ready time, index) if nothing queued is running and it fits.
    M admitted = 0;
    if (qfin <= t) {
      const M qw = ~started & gqm & ALL;
      uint32_t hT = kInf, hmem = 0;
      M hbit = 0;
#pragma unroll
      for (int v = 0; v < N; ++v) {
        if (bit<N>(qw, v) && T[v] <= t && T[v] < hT) {
          hT = T[v];
          hbit = M(1) << v;
          hmem = tab[kHdrWords + kToolWords * v + kToolMem];
        }
      }
      if (hbit != 0 && hmem <= budget - in_use) {
        admitted = hbit;
        k += 1;
      }
    }
    st |= admitted;

    // Durations of everything starting at t.
    const uint32_t lev = umin32(umax32(k, 1u), levels) - 1u;
#pragma unroll
    for (int v = 0; v < N; ++v) {
      if (bit<N>(st, v)) {
        uint32_t d;
        if (bit<N>(gpum, v))
          d = s_dur[(uint32_t(v) * 2u + uint32_t(bit<N>(gqm, v))) * levels + lev];
        else
          d = tab[kHdrWords + kToolWords * v + kToolCpu];
        T[v] = t + d;
        if (bit<N>(admitted, v)) qfin = T[v];
      }
    }
    started |= st;
    if (started == ALL) {
      uint32_t ms = 0;
#pragma unroll
      for (int v = 0; v < N; ++v) ms = umax32(ms, T[v]);
      result = ms;
      break;
    }

    // Ready times of waiting tools whose predecessors have all started:
    // r_w = max over u -> w of C_u (+ xfer_w when u and w sit on different
    // devices).  Predecessor lists are wave-uniform; T[u] is read with a
    // uniform register index.
#pragma unroll
    for (int w = 0; w < N; ++w) {
      const uint32_t* rec = tab + kHdrWords + kToolWords * w;
      const M pm = load_mask<N>(rec, kToolPredLo);
      if (!bit<N>(started, w) && T[w] == kInf && (pm & ~started) == 0) {
        const uint32_t np = rec[kToolNPred];
        const uint32_t* pl = tab + kPredBase + rec[kToolPredOff];
        const uint32_t xw = rec[kToolXfer];
        const bool gw = bit<N>(gpum, w);
        uint32_t r = 0;
        for (uint32_t j = 0; j < np; ++j) {
          const int u = DEVMAP_UNIFORM(int(pl[j]));
          const uint32_t arrive = T[u] + ((bit<N>(gpum, u) != gw) ? xw : 0u);
          r = umax32(r, arrive);
        }
        T[w] = r;
      }
    }

    // Next event: the smallest ready or finish time after t.
    uint32_t tn = kInf;
#pragma unroll
    for (int v = 0; v < N; ++v) tn = umin32(tn, T[v] > t ? T[v] : kInf);
    if (tn == kInf) break;  // a queued tool can never fit: infeasible
    t = tn;
  }
  return result;
}

// Decode tools lo_tool..N-1 of x (x = their base-3 digits, lowest first)
// into mode masks.
template <int N>
__host__ __device__ __forceinline__ void decode_digits(uint64_t x, int lo_tool, MaskT<N>& gn,
                                              MaskT<N>& gq) {
  using M = MaskT<N>;
  gn = 0;
  gq = 0;
  if (x < (1ull << 32)) {
    uint32_t y = uint32_t(x);
    for (int v = lo_tool; v < N; ++v) {
      const uint32_t q = y / 3u, d = y - 3u * q;
      if (d == 1) gn |= M(1) << v;
      if (d == 2) gq |= M(1) << v;
      y = q;
    }
  } else {
    for (int v = lo_tool; v < N; ++v) {
      const uint64_t q = x / 3u;
      const uint32_t d = uint32_t(x - 3u * q);
      if (d == 1) gn |= M(1) << v;
      if (d == 2) gq |= M(1) << v;
      x = q;
    }
  }
}

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

template <int N>
__device__ __forceinline__ void stage_durations(const uint32_t* tab, uint32_t* s_dur) {
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t* dur = tab + tab[kHdrDurOff];
  for (uint32_t i = threadIdx.x; i < uint32_t(N) * 2u * levels; i += blockDim.x) s_dur[i] = dur[i];
  __syncthreads();
}

// One lane's share of one work item: outer combination
// outer_lo + item * kBlock + lane (the modes of tools J..N-1), combined with
// every inner combination (tools 0..J-1) whose index lies in [lo, hi).
// Updates the lane's running (makespan, index) minimum; indices are visited
// in increasing order, so a strict comparison keeps the lowest index.
template <int N>
__host__ __device__ __forceinline__ void lane_search(const SearchArgs& a,
                                                     const uint32_t* __restrict__ tab,
                                                     const uint32_t* __restrict__ s_dur,
                                                     uint64_t item, uint32_t lane,
                                                     uint32_t& best_ms, uint64_t& best_x) {
  using M = MaskT<N>;
  const uint64_t rel = item * kBlock + lane;
  if (rel >= a.n_outer) return;
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t budget = tab[kHdrBudget];
  const uint32_t J = a.inner_digits;
  const uint64_t o = a.outer_lo + rel;
  M ogn, ogq;
  decode_digits<N>(o, int(J), ogn, ogq);  // o's digits are tools J..N-1
  const uint64_t base = o * a.inner_count;
  // Inner index bounds of this lane inside [lo, hi).
  const uint64_t ilo64 = a.lo > base ? a.lo - base : 0;
  const uint64_t ihi64 = a.hi - base;  // > 0 because o < ceil(hi / 3^J)
  const uint32_t ilo = uint32_t(ilo64 < a.inner_count ? ilo64 : a.inner_count);
  const uint32_t ihi = uint32_t(ihi64 < a.inner_count ? ihi64 : a.inner_count);
  M ign = 0, igq = 0;  // inner modes: the same in every lane of the wave
  for (uint32_t i = 0; i < a.inner_count; ++i) {
    if (i >= ilo && i < ihi) {
      const uint32_t ms = evaluate<N>(tab, s_dur, levels, budget, ogn | ign, ogq | igq);
      if (ms < best_ms) {
        best_ms = ms;
        best_x = base + i;
      }
    }
    // odometer step on the inner digits
    M b = 1;
    for (uint32_t j = 0; j < J; ++j, b <<= 1) {
      if (igq & b) {
        igq &= ~b;
        continue;
      }
      if (ign & b) {
        ign &= ~b;
        igq |= b;
      } else {
        ign |= b;
      }
      break;
    }
  }
}

// Exhaustive search.  Block b serves table b / blocks_per_table and walks its
// work items (kBlock consecutive outer combinations each) with a stride of
// blocks_per_table.  Each lane keeps its own (makespan, index) minimum; the
// block's minimum goes to partials[b].
template <int N>
__global__ __launch_bounds__(kBlock) void search_kernel(SearchArgs a) {
  __shared__ uint32_t s_dur[N * 2 * (N < kMaxLevels ? N : kMaxLevels)];
  const uint32_t table = blockIdx.x / a.blocks_per_table;
  const uint32_t bb = blockIdx.x - table * a.blocks_per_table;
  const uint32_t* tab = a.tables + size_t(table) * a.table_stride;
  stage_durations<N>(tab, s_dur);

  uint32_t best_ms = kInf;
  uint64_t best_x = ~0ull;
  for (uint64_t item = bb; item < a.items_per_table; item += a.blocks_per_table)
    lane_search<N>(a, tab, s_dur, item, threadIdx.x, best_ms, best_x);

  block_min(best_ms, best_x);
  if (threadIdx.x == 0) {
    Partial p;
    p.index = best_x;
    p.makespan = best_ms;
    p.pad = 0;
    a.partials[blockIdx.x] = p;
  }
}

// Score explicit indices (grid-stride).
template <int N>
__global__ __launch_bounds__(kBlock) void eval_kernel(const uint32_t* __restrict__ tab,
                                                      const uint64_t* __restrict__ idx,
                                                      int64_t n, uint64_t n_mappings,
                                                      int64_t* __restrict__ out) {
  using M = MaskT<N>;
  __shared__ uint32_t s_dur[N * 2 * (N < kMaxLevels ? N : kMaxLevels)];
  stage_durations<N>(tab, s_dur);
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t budget = tab[kHdrBudget];
  for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kBlock) {
    const uint64_t x = idx[i];
    int64_t r = INT64_MAX;
    if (x < n_mappings) {
      M gn, gq;
      decode_digits<N>(x, 0, gn, gq);
      const uint32_t ms = evaluate<N>(tab, s_dur, levels, budget, gn, gq);
      if (ms != kInf) r = int64_t(ms);
    }
    out[i] = r;
  }
}

// Launchers of one instantiation (explicitly instantiated per tool count in
// the inst_*.hip translation units).
template <int N>
hipError_t launch_search_n(const SearchArgs& a, hipStream_t s) {
  const uint32_t blocks = a.n_tables * a.blocks_per_table;
  hipLaunchKernelGGL(search_kernel<N>, dim3(blocks), dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

template <int N>
hipError_t launch_eval_n(const uint32_t* tab, const uint64_t* idx, int64_t n,
                                uint64_t n_mappings, int64_t* out, hipStream_t s) {
  int64_t blocks = (n + kBlock - 1) / kBlock;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(eval_kernel<N>, dim3(uint32_t(blocks)), dim3(kBlock), 0, s, tab, idx, n,
                     n_mappings, out);
  return hipGetLastError();
}

}  // namespace devmap
