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
#include "reduce.h"

namespace devmap {

template <int N>
using MaskT = typename std::conditional<(N <= 32), uint32_t, uint64_t>::type;

// Read-only view of a problem table.  On the device it reads through the
// constant address space, so wave-uniform reads become scalar loads.
struct Tab {
  const uint32_t* p;
  __host__ __device__ __forceinline__ uint32_t operator[](uint32_t i) const {
#if defined(__HIP_DEVICE_COMPILE__)
    typedef const __attribute__((address_space(4))) uint32_t* ConstPtr;
    return ((ConstPtr)p)[i];
#else
    return p[i];
#endif
  }
  __host__ __device__ __forceinline__ Tab operator+(uint32_t i) const { return Tab{p + i}; }
};

// The table, opaque to the optimiser: reads through the returned view are
// re-issued where they are used (scalar-cache hits) instead of being hoisted
// out of the event loop into registers that would then spill.
__host__ __device__ __forceinline__ Tab fresh(const uint32_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+s"(p));
#endif
  return Tab{p};
}

// A wave-uniform value the optimiser must not carry across this point: its
// bit tests are recomputed in scalar registers where they are used rather
// than kept live as lane masks (which would crowd the scalar register file).
template <class M>
__host__ __device__ __forceinline__ M opaque(M x) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+s"(x));
#endif
  return x;
}

// An empty side effect: keeps a wave-uniform branch a branch instead of
// letting the optimiser turn its body into per-lane selects.
#if defined(__HIP_DEVICE_COMPILE__)
#define DEVMAP_KEEP_BRANCH() asm volatile("")
#else
#define DEVMAP_KEEP_BRANCH() ((void)0)
#endif

__host__ __device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }
__host__ __device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }
// max(g, f) over GPU finishes only, for g >= 0: a GPU finish lies below 2^30
// (positive as a signed word), a CPU finish carries the top tag bits
// (negative), so one signed maximum leaves g as it is for the latter.
__host__ __device__ __forceinline__ uint32_t smax_gpu(uint32_t g, uint32_t f) {
  const int32_t a = int32_t(g), b = int32_t(f);
  return uint32_t(a > b ? a : b);
}

// c ? acc + x : acc (and c ? acc | x : acc) as an add (or) and one select.
// The sum is formed first, opaque to the optimiser, so that a wave-uniform x
// enters the add directly instead of being moved to a vector register for a
// select of x or 0.
__host__ __device__ __forceinline__ uint32_t add_if(uint32_t acc, uint32_t x, bool c) {
  uint32_t s = acc + x;
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(s));
#endif
  return c ? s : acc;
}
// A per-lane value the optimiser must not carry across this point.
template <class M>
__host__ __device__ __forceinline__ M opaque_v(M x) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(x));
#endif
  return x;
}

template <class M>
__host__ __device__ __forceinline__ M or_if(M acc, M x, bool c) {
  M s = acc | x;
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(s));
#endif
  return c ? s : acc;
}

template <int N>
__host__ __device__ __forceinline__ MaskT<N> all_tools() {
  if constexpr (N == 32) return 0xFFFFFFFFu;
  else if constexpr (N == 64) return ~0ull;
  else return (MaskT<N>(1) << N) - 1;
}

template <int N, class P>
__host__ __device__ __forceinline__ MaskT<N> load_mask(const P& tab, uint32_t lo_word) {
  if constexpr (N <= 32) return tab[lo_word];
  else return uint64_t(tab[lo_word]) | (uint64_t(tab[lo_word + 1]) << 32);
}

template <int N>
__host__ __device__ __forceinline__ bool bit(MaskT<N> m, int v) {
  return (m >> v) & 1;
}

// LDS image staged by every block: footprints by internal label, then the
// duration table (its length follows the problem's contention levels),
// level-major:
// dur[(level - 1) * 2N + 2 * label + q] (q = 0 gpu_now, 1 gpu_queue), so a
// pass finds its row once and each start reads one word at a fixed offset.
template <int N>
constexpr uint32_t lds_levels() { return N < kMaxLevels ? N : kMaxLevels; }
template <int N>
constexpr uint32_t lds_mem_off() { return 0u; }
template <int N>
constexpr uint32_t lds_dur_off() { return uint32_t(N); }
// Words of the image for `levels` stored contention levels.
__host__ __device__ constexpr uint32_t lds_words_for(int n, uint32_t levels) {
  return uint32_t(n) + uint32_t(n) * 2u * levels;
}
// The largest image a problem with N tools can need.
template <int N>
constexpr uint32_t lds_words() { return lds_words_for(N, lds_levels<N>()); }

// Bitwise OR of x over the active lanes of the calling wave, through one LDS
// word per wave (slot).  Lanes that have left the calling loop simply do not
// contribute, so the result is right under divergence too.  A host build has
// one lane per "wave": the result is x itself.
template <class M>
__host__ __device__ __forceinline__ M wave_or(M x, M* slot) {
#if defined(__HIP_DEVICE_COMPILE__)
  __hip_atomic_store(slot, M(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
  __builtin_amdgcn_wave_barrier();
  __hip_atomic_fetch_or(slot, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
  __builtin_amdgcn_wave_barrier();
  const M r = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
  __builtin_amdgcn_wave_barrier();
  if constexpr (sizeof(M) == 4) {
    return __builtin_amdgcn_readfirstlane(r);
  } else {
    // (the builtin returns a signed word: each half is taken back as
    // unsigned before widening, or a low word with bit 31 set would fill the
    // high word with ones)
    return (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(r >> 32)))) << 32) |
           uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(r))));
  }
#else
  (void)slot;
  return x;
#endif
}

// Wave-wide OR of three per-lane tool masks through the calling wave's 8-byte
// LDS slot: one 64-bit OR when 3N bits fit, else one per mask (or pair).
template <int N>
__host__ __device__ __forceinline__ void wave_or3(MaskT<N> a, MaskT<N> b, MaskT<N> c,
                                                  MaskT<N>* slot, MaskT<N>& oa, MaskT<N>& ob,
                                                  MaskT<N>& oc) {
  using M = MaskT<N>;
  uint64_t* const s64 = reinterpret_cast<uint64_t*>(slot);
  if constexpr (3 * N <= 64) {
    constexpr uint64_t m = (uint64_t(1) << N) - 1u;
    const uint64_t r = wave_or<uint64_t>(uint64_t(a) | (uint64_t(b) << N) | (uint64_t(c) << (2 * N)),
                                         s64);
    oa = M(r & m);
    ob = M((r >> N) & m);
    oc = M((r >> (2 * N)) & m);
  } else if constexpr (N <= 32) {
    const uint64_t r = wave_or<uint64_t>(uint64_t(a) | (uint64_t(b) << 32), s64);
    oa = M(r);
    ob = M(r >> 32);
    oc = wave_or<uint64_t>(uint64_t(c), s64);
  } else {
    oa = wave_or<M>(a, slot);
    ob = wave_or<M>(b, slot);
    oc = wave_or<M>(c, slot);
  }
}

// Event-driven schedule of one mapping (the schedule model in full), advanced
// one event time per call of step().
//
// gnm / gqm: tools on gpu_now / gpu_queue (internal labels; the rest run on
// the CPU).  A tool is first unresolved, then waiting (its ready time is
// known), then started (its finish time is known); it never needs both times
// at once, so one register T[i] per tool holds its state.  Times stay below
// H = 2^30 (a creation-time guard), which leaves the two top bits as a tag:
//   0            unresolved
//   f            started on the GPU, finishing at f (f >= 1)
//   H + r        waiting gpu_now tool, ready at r
//   2H + r       waiting gpu_queue tool, ready at r
//   3H + f       CPU tool finishing at f
// One unsigned difference then answers each question: a GPU tool runs at t
// iff T - (t+1) < H - (t+1); a queued tool is ready iff T - 2H <= t; and so on.
// A CPU tool starts the moment its inputs arrive and neither slows nor blocks
// anything, so it is resolved as soon as all its predecessors have started;
// the ascending sweep over topological labels resolves chains of CPU tools
// in one pass.  Pass 0 only resolves the sources; every later pass handles
// one event time t:
//   A. GPU tools running at t plus gpu_now tools ready at t give the
//      concurrency k and the VRAM in use (over the budget: out of memory);
//      if no queued tool is running and one is ready, the queue head -- the
//      lowest original number among the queued tools ready at minq, the
//      earliest ready time -- is admitted when it fits;
//   B. in label order: starters get f = t + dur[k], fixed for their life;
//      tools whose predecessors have all started get their ready time
//      r = max over u -> i of finish(u) (+ xfer_i across devices); and the
//      next event is chosen: the next gpu_now ready time, and while a ready
//      queued tool waits, the queue's finish (busy queue) or the next GPU
//      finish (VRAM); otherwise the next queued ready time.  While the head
//      waits, a later queued arrival cannot move it, so that time is no
//      event (visiting it would change nothing).
// A pass visits a tool only where some lane of the wave needs it, by the
// tool's state there: waiting (resolved, not started), running (a GPU tool
// running at the previous event, or started there) or unresolved -- three
// wave-wide ORs.  The work of a tool in any other state would change
// nothing, so skipping it changes no result.  A tool's next-event
// contribution is taken where its time becomes known (its start or its
// resolution) or from its state.
// A mapping needs at most 2N+1 passes: every pass after the first moves t to
// a ready or finish time, and each tool has one of each.
constexpr uint32_t kH = 0x40000000u;  // 2^30: time limit and tag unit
constexpr uint32_t kTagNow = kH;
constexpr uint32_t kTagQueue = 2u * kH;
constexpr uint32_t kTagCpu = 3u * kH;

template <int N>
struct Sim {
  using M = MaskT<N>;
  uint32_t T[N];
  M gnm, gqm;
  M started;   // started GPU tools and resolved CPU tools
  M resolved;  // tools whose ready time is known
  M run;       // GPU tools running at the last pass's t or started there
  uint32_t t;
  uint32_t qfin;  // finish of the running queued tool (0: none)
  uint32_t minq;  // earliest ready time of a waiting queued tool (>= H: none)
  uint32_t mk;    // latest finish of the started tools
  uint32_t rgs;   // deferred tools: earliest ready time on the GPU (kInf: none known)
  bool dead;      // statically infeasible

  __host__ __device__ __forceinline__ void init(const uint32_t* __restrict__ tab, M gn, M gq) {
    gnm = gn;
    gqm = gq;
#pragma unroll
    for (int i = 0; i < N; ++i) T[i] = 0;
    started = 0;
    resolved = 0;
    run = 0;
    t = 0;
    qfin = 0;
    minq = kInf;
    mk = 0;
    rgs = kInf;
    // a GPU mode whose footprint exceeds the budget never fits
    dead = ((gn | gq) & load_mask<N>(Tab{tab}, kHdrBigLo)) != 0;
  }

  // Pass number `pass` (wave-uniform: the lanes of a wave start their
  // mappings together).  Returns true when the mapping is settled; ms then
  // holds its makespan, or kInf if it is infeasible.  slot: this wave's LDS
  // word for the wave-wide masks.
  //
  // DEFER (schedule prefixes shared by the modes of `defer`, a wave-uniform
  // set of sinks that have predecessors): a deferred tool's mode is never
  // read.  When its predecessors have all started it is marked resolved and
  // started with T = 0, which keeps it out of every later per-tool loop, and
  // its ready time on the GPU joins rgs, which is an event.  Before that
  // time the tool cannot run, hold VRAM, queue or feed a successor in any
  // mode (and on the CPU it only adds its own finish to the makespan), so
  // the passes before rgs are those of every mode.  Once a deferred tool is
  // resolved a pass ends the mapping only as infeasible; the caller stops at
  // t == rgs.
  template <bool DEFER = false>
  __host__ __device__ __forceinline__ bool step(const uint32_t* __restrict__ tab,
                                                const uint32_t* __restrict__ lds,
                                                uint32_t levels, uint32_t budget, int pass,
                                                M* slot, uint32_t& ms, M defer = 0) {
    ms = kInf;
    if (dead) return true;
    // the modes, re-read each pass: tests of these loop-invariant lane masks
    // would otherwise be hoisted out of the event loop as one scalar mask
    // pair per tool, more than the scalar registers hold
    gnm = opaque_v(gnm);
    gqm = opaque_v(gqm);
    const M ALL = all_tools<N>();
    const M gpum = gnm | gqm;
    const uint32_t* s_dur = lds + lds_dur_off<N>();
    const uint32_t* s_mem = lds + lds_mem_off<N>();
    const Tab tp = fresh(tab);
    const uint32_t t1 = t + 1u;
    const uint32_t lim = kH - t1;  // d = x - t1 < lim: x is a time after t
    const uint32_t now_t = kTagNow + t;
    // tools some lane of the wave has waiting / running / unresolved
    M ww, wr, wu;
    wave_or3<N>(resolved & ~started, run, ALL & ~resolved, slot, ww, wr, wu);

    // A. concurrency and VRAM at t, after releases and immediate starts; the
    // earliest finish after t of a running tool; the queue head.  One loop
    // over the tools running or waiting in some lane, one test for a tool in
    // neither state: fewer scalar instructions and table reads than a loop
    // per state.
    uint32_t in_use = 0, k = 0, tf = kInf;
    run = 0;
    // the queue head, if the queue is free and a queued tool ready: ready at
    // minq (the earliest), lowest original number (the table's word holds
    // the number above the label)
    const bool qfree = minq <= t && qfin <= t;
    // (formed once: the tag is the top bit, and a compare against the sum
    // would otherwise become a per-tool flip of T's top bit)
    const uint32_t key = opaque_v(kTagQueue + minq);
    uint32_t hO = kInf;
    const M wr_a = opaque(wr), ww_a = opaque(ww), wa_a = opaque(wr | ww);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (!((wa_a >> i) & 1)) continue;  // one test for a tool in neither state
      DEVMAP_KEEP_BRANCH();
      const uint32_t mem = opaque(tp[kHdrWords + kToolWords * i + kToolMem]);
      if ((wr_a >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        const uint32_t d = T[i] - t1;
        const bool on = d < lim;  // finishes after t
        in_use = add_if(in_use, mem, on);
        run = or_if(run, M(1) << i, on);
        tf = umin32(tf, d);
      }
      if ((ww_a >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        const bool on = T[i] == now_t;  // gpu_now, ready at t
        in_use = add_if(in_use, mem, on);
        k += on ? 1u : 0u;
        const uint32_t orig = opaque(tp[kHdrWords + kToolWords * i + kToolOrig]);
        hO = T[i] == key ? umin32(hO, orig) : hO;  // read only if qfree
      }
    }
    if constexpr (N <= 32) {
      k += __builtin_popcount(uint32_t(run));
    } else {
      k += __builtin_popcountll(uint64_t(run));
    }
    if (in_use > budget) return true;  // out of memory: infeasible
    uint32_t hsel = kInf;              // label of the queued tool admitted at t
    if (qfree) {
      const uint32_t lab = hO & kOrigLabelMask;
      if (s_mem[lab] <= budget - in_use) {
        hsel = lab;
        k += 1;
      }
    }
    const uint32_t lev = umin32(umax32(k, 1u), levels) - 1u;
    const uint32_t* const s_row = s_dur + lev * (2u * uint32_t(N));  // durations at level lev + 1

    // B. starts, resolution, next event (waiting and unresolved tools)
    const uint32_t now_t1 = opaque_v(now_t + 1u);  // formed once, not per tool
    uint32_t tn = kInf;
    minq = kInf;
    const M ww_b = opaque(ww), wu_b = opaque(wu), wb_b = opaque(ww | wu);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const M bi = M(1) << i;
      if (!((wb_b >> i) & 1)) continue;  // one test for a tool in neither state
      DEVMAP_KEEP_BRANCH();
      if ((ww_b >> i) & 1) {
        const bool adm = (hsel == uint32_t(i));
        if (T[i] == now_t || adm) {
          const uint32_t d = s_row[2u * uint32_t(i) + (adm ? 1u : 0u)];
          T[i] = t + d;
          started |= bi;
          run |= bi;
          tf = umin32(tf, d - 1u);  // finish after t
          mk = umax32(mk, T[i]);
          if (adm) qfin = T[i];
        }
        const uint32_t x = T[i];
        tn = umin32(tn, x - now_t1);           // gpu_now ready after t
        minq = umin32(minq, x - kTagQueue);   // queued ready time (>= H: none)
      }
      if ((wu_b >> i) & 1) {
        const M pm = load_mask<N>(tp, kHdrWords + kToolWords * i + kToolPredLo);
        if (T[i] == 0 && (started & pm) == pm) {
          const Tab rec = fresh(tab) + (kHdrWords + kToolWords * i);
          uint32_t g = 0, c = 0;  // latest GPU finish; latest finish overall
          // Predecessors carry smaller labels; the mask test is wave-uniform.
#pragma unroll
          for (int u = 0; u < i; ++u) {
            if ((pm >> u) & 1) {  // scalar branch: no vector work for non-edges
              DEVMAP_KEEP_BRANCH();
              const uint32_t f = T[u];
              g = smax_gpu(g, f);
              c = umax32(c, f);  // CPU finishes carry the top tag, so they dominate
            }
          }
          c = c >= kTagCpu ? c - kTagCpu : 0u;  // latest CPU finish (0: none)
          const uint32_t xw = rec[kToolXfer];
          const uint32_t rg = umax32(g, c ? c + xw : 0u);  // ready time on the GPU
          resolved |= bi;
          if (DEFER && ((defer >> i) & 1)) {
            // prefix: modes of deferred tools are CPU, so the GPU ready time
            // needs its own expression
            rgs = umin32(rgs, rg);
            started |= bi;
          } else {
            // selects, not branches: the modes are per lane
            const bool on_gpu = (gpum >> i) & 1, now = (gnm >> i) & 1;
            const uint32_t f = umax32(c, g ? g + xw : 0u) + rec[kToolCpu];  // CPU finish
            T[i] = on_gpu ? (now ? kTagNow : kTagQueue) + rg : kTagCpu + f;
            started = or_if(started, bi, !on_gpu);
            mk = on_gpu ? mk : umax32(mk, f);
            // the next-event terms of the waiting tools, from the tagged
            // word: outside its own mode a term lands at or above the range
            // it is read in (as in the sweep over waiting tools)
            tn = umin32(tn, T[i] - now_t1);
            minq = umin32(minq, T[i] - kTagQueue);
          }
        }
      }
    }
    if (started == ALL && (!DEFER || rgs == kInf)) {
      ms = mk;
      return true;
    }
    if (pass == 0) return false;  // sources resolved: now the events at t = 0
    uint32_t next = kInf;
    if (tn < lim) next = tn + t1;
    if (minq <= t) {
      // A ready queued tool is still waiting: the queue head can only move
      // when the queue frees or VRAM is released, whatever else turns ready.
      if (qfin > t) {
        next = umin32(next, qfin);     // queue busy: wait for it
      } else if (tf < lim) {
        next = umin32(next, tf + t1);  // blocked on VRAM: wait for a release
      }
    } else if (minq < kH) {
      next = umin32(next, minq);       // the next queued tool turns ready
    }
    if (DEFER) next = umin32(next, rgs);
    if (next == kInf) return true;  // a queued tool can never fit: infeasible
    t = next;
    return false;
  }

  // After a DEFER prefix stopped at t == rgs, with the modes now set: give
  // every deferred tool the prefix resolved the state the resolution step
  // would have given it (its predecessors have all started, so their
  // finishes are final).  Deferred tools still unresolved stay so, and the
  // ordinary passes resolve them.
  __host__ __device__ __forceinline__ void settle_deferred(const uint32_t* __restrict__ tab,
                                                           M defer) {
    const M gpum = gnm | gqm;
    const Tab tp = fresh(tab);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if ((defer >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        const M bi = M(1) << i;
        if (resolved & bi) {
          const M pm = load_mask<N>(tp, kHdrWords + kToolWords * i + kToolPredLo);
          uint32_t g = 0, c = 0;
#pragma unroll
          for (int u = 0; u < i; ++u) {
            if ((pm >> u) & 1) {
              DEVMAP_KEEP_BRANCH();
              const uint32_t f = T[u];
              g = smax_gpu(g, f);
              c = umax32(c, f);
            }
          }
          c = c >= kTagCpu ? c - kTagCpu : 0u;
          const Tab rec = tp + (kHdrWords + kToolWords * i);
          const uint32_t xw = rec[kToolXfer];
          const bool on_gpu = (gpum & bi) != 0;
          const uint32_t r = on_gpu ? umax32(g, c ? c + xw : 0u) : umax32(c, g ? g + xw : 0u);
          if (!on_gpu) {
            const uint32_t f = r + rec[kToolCpu];
            T[i] = kTagCpu + f;
            mk = umax32(mk, f);
          } else {
            started &= ~bi;
            if (gnm & bi) {
              T[i] = kTagNow + r;
            } else {
              T[i] = kTagQueue + r;
              minq = umin32(minq, r);
            }
          }
        }
      }
    }
  }
};

// Makespan of one mapping of a fan-out whose footprints all fit the budget
// together (kFlagFreeFanout), fixed-at-start contention.  Every tool is ready
// at 0.  The CPU tools end at their cpu_us.  The gpu_now tools and the first
// queued tool (the lowest number: the queue orders ties by number) start at
// 0 with k0 = #gpu_now + 1 co-running GPU tools (k0 = #gpu_now with an empty
// queue), and the queue never waits for VRAM, so each later queued tool
// starts when its predecessor in the queue ends, at s, beside the gpu_now
// tools still running (finish > s: releases come first) and itself.  No other
// event changes a duration.  Labels are tool numbers.  slot: the calling
// wave's LDS word (see wave_or).
template <int N>
__host__ __device__ __forceinline__ uint32_t evaluate_fanout(const uint32_t* __restrict__ tab,
                                                             const uint32_t* __restrict__ lds,
                                                             uint32_t levels, MaskT<N> gnm,
                                                             MaskT<N> gqm, MaskT<N>* slot) {
  using M = MaskT<N>;
  const uint32_t* s_dur = lds + lds_dur_off<N>();
  constexpr uint32_t kRow = 2u * uint32_t(N);
  const Tab tp = fresh(tab);
  // tools some lane of the wave has on gpu_now / gpu_queue
  M wn, wq, wx;
  wave_or3<N>(gnm, gqm, M(0), slot, wn, wq, wx);
  uint32_t k0;
  if constexpr (N <= 32) {
    k0 = uint32_t(__builtin_popcount(uint32_t(gnm)));
  } else {
    k0 = uint32_t(__builtin_popcountll(uint64_t(gnm)));
  }
  k0 += gqm != 0 ? 1u : 0u;
  const uint32_t* row0 = s_dur + (umin32(umax32(k0, 1u), levels) - 1u) * kRow;
  uint32_t f[N];  // finish of each gpu_now tool (0 for the others)
  uint32_t mk = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    f[i] = 0;
    if ((wn >> i) & 1) {
      DEVMAP_KEEP_BRANCH();
      if ((gnm >> i) & 1) f[i] = row0[2 * i];
    }
    const bool cpu = !(((gnm | gqm) >> i) & 1);
    mk = umax32(mk, cpu ? opaque(tp[kHdrWords + kToolWords * i + kToolCpu]) : f[i]);
  }
  const M wn_q = opaque(wn), wq_q = opaque(wq);
  uint32_t s = 0;  // when the queue frees
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if ((wq_q >> i) & 1) {
      DEVMAP_KEEP_BRANCH();
      if ((gqm >> i) & 1) {
        uint32_t k = 1;
#pragma unroll
        for (int v = 0; v < N; ++v) {
          if ((wn_q >> v) & 1) {
            DEVMAP_KEEP_BRANCH();
            k += f[v] > s ? 1u : 0u;
          }
        }
        s += s_dur[(umin32(k, levels) - 1u) * kRow + 2u * uint32_t(i) + 1u];
        mk = umax32(mk, s);
      }
    }
  }
  return mk;
}

// Makespan of one mapping, or kInf if it is infeasible.  slot: the calling
// wave's LDS word (see wave_or).
template <int N>
__host__ __device__ __forceinline__ uint32_t evaluate(const uint32_t* __restrict__ tab,
                                                      const uint32_t* __restrict__ lds,
                                                      uint32_t levels, uint32_t budget,
                                                      MaskT<N> gnm, MaskT<N> gqm,
                                                      MaskT<N>* slot) {
  if (Tab{tab}[kHdrFlags] & kFlagFreeFanout)
    return evaluate_fanout<N>(tab, lds, levels, gnm, gqm, slot);
  Sim<N> sim;
  sim.init(tab, gnm, gqm);
  uint32_t ms = kInf;
  for (int pass = 0; pass < 2 * N + 2; ++pass)
    if (sim.step(tab, lds, levels, budget, pass, slot, ms)) break;
  return ms;
}

// High 64 bits of the 128-bit product x * y.
__host__ __device__ __forceinline__ uint64_t mulhi64(uint64_t x, uint64_t y) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __umul64hi(x, y);
#else
  return uint64_t((unsigned __int128)x * y >> 64);
#endif
}

// ceil(a / w) for a < 2^46 and 256 <= w <= 2^16, in integers only, with
// winv = floor(2^48 / w) from the table: a * winv / 2^48 lies within a
// quarter below a / w, so its floor is the quotient or one less, and one
// remainder step makes it exact.
__host__ __device__ __forceinline__ uint64_t ceil_div_small(uint64_t a, uint32_t w,
                                                           uint64_t winv) {
  uint64_t q = mulhi64(a << 16, winv);
  uint64_t r = a - q * w;
  if (r >= w) {
    q += 1;
    r -= w;
  }
  return q + (r != 0 ? 1u : 0u);
}

// Event loop under processor sharing, one event time per call of step().
// The events are those of the fixed-at-start schedule (release, immediate
// starts with the VRAM check, one queue admission in (ready, tool) order),
// but a GPU task's end is not fixed when it starts: every running GPU task
// advances at the rate w_k of the k GPU tasks running, so with V the work
// each has done since time 0, a task started at V_s with work b * 2^16 ends
// when V reaches its virtual finish V_s + b * 2^16.  A CPU task neither
// slows nor blocks anything and starts at its ready time, so it is resolved
// (started, its end known) as soon as the ends of all its predecessors are
// known, in one ascending sweep over the labels; its end is then no event.
// A tool's ready time is computed once, when its predecessors' ends are all
// known: a CPU predecessor's when it is resolved, a GPU predecessor's when it
// is done.  Each per-tool loop visits a tool only where some lane of the wave
// has it running or not yet started (two wave-wide ORs per pass); elsewhere
// its work would change nothing.  A tool's mode is first read when its ready
// time is computed (first_read: resolved | cpu).
template <int N>
struct SimPS {
  using M = MaskT<N>;
  // Y[i]: the virtual finish of a running GPU task, else (low word) its
  // ready time while waiting and its end once started or done
  uint64_t Y[N];
  M gnm, gqm;
  M running, done;  // GPU tasks
  M resolved;       // GPU tasks whose ready time is known
  M cpu;            // CPU tasks, resolved: started at their ready time, end known
  uint64_t V;
  uint32_t t;
  uint32_t mk;   // latest end of the CPU tasks
  uint32_t rgs;  // deferred tools: earliest ready time on the GPU (kInf: none known)
  bool dhit;     // a deferred tool's GPU ready time came due in the last pass
  bool dead;     // statically infeasible

  __host__ __device__ __forceinline__ void init(const uint32_t* __restrict__ tab, M gn, M gq) {
    gnm = gn;
    gqm = gq;
#pragma unroll
    for (int i = 0; i < N; ++i) Y[i] = 0;
    running = 0;
    done = 0;
    resolved = 0;
    cpu = 0;
    V = 0;
    t = 0;
    mk = 0;
    rgs = kInf;
    dhit = false;
    dead = ((gn | gq) & load_mask<N>(Tab{tab}, kHdrBigLo)) != 0;
  }

  // One event time.  Returns true when the mapping is settled; ms then holds
  // its makespan, or kInf if it is infeasible.
  //
  // DEFER (schedule prefixes shared by the modes of `defer`, a wave-uniform
  // set of sinks with predecessors, which the prefix runs on the CPU): once
  // the ends of a deferred tool's predecessors are known it is parked (in
  // `cpu`, end unknown, excluded from the makespan) and its ready time on the
  // GPU joins rgs, an event; until then it cannot run, hold VRAM, queue or
  // feed a successor in any mode.  If that ready time is not after t, the
  // pass has handled events at which the tool could already act: dhit tells
  // the caller to restart the pass from the state before it.
  template <bool DEFER = false>
  __host__ __device__ __forceinline__ bool step(const uint32_t* __restrict__ tab,
                                                const uint32_t* __restrict__ lds,
                                                uint32_t levels, uint32_t budget, int pass,
                                                M* slot, uint32_t& ms, M defer = 0) {
    (void)pass;
    ms = kInf;
    if (dead) return true;
    // the modes and the tool records, re-read each pass (see Sim::step): the
    // tests of loop-invariant values would otherwise be hoisted out of the
    // event loop as scalar lane masks, more than the scalar registers hold
    gnm = opaque_v(gnm);
    gqm = opaque_v(gqm);
    const Tab tp = fresh(tab);
    const uint32_t* s_mem = lds + lds_mem_off<N>();
    const uint32_t* sh = tab + tab[kHdrShareOff];
    const M gpu = gnm | gqm;
    const M ALL = all_tools<N>();
    // tools some lane of the wave has running / not yet started
    M wr, ww;
    if constexpr (N <= 32) {
      const uint64_t both = wave_or<uint64_t>(
          uint64_t(running) | (uint64_t(ALL & ~(running | done | cpu)) << 32),
          reinterpret_cast<uint64_t*>(slot));
      wr = M(both);
      ww = M(both >> 32);
    } else {
      wr = wave_or<M>(running, slot);
      ww = wave_or<M>(ALL & ~(running | done | cpu), slot);
    }
    // 1. release: GPU tasks out of work; VRAM and least virtual finish of
    // those still running.  2. ready times of tasks whose predecessors' ends
    // are all known (CPU tasks start there), the immediate GPU starts, and
    // the ready times still to come (events).  3. the queue head.  One sweep
    // in label order over the tools running or not yet started in some lane:
    // a predecessor (a lower label) is released before its successor is
    // examined.
    uint32_t in_use = 0;
    uint32_t next = kInf;  // the next event: ready times after t (GPU ends follow below)
    uint64_t vmin = ~0ull;  // the least virtual finish of the GPU tasks running after t
    M starting = 0;
    uint64_t hk = ~0ull;  // the lowest (ready time, original number) of a ready queued task
    const M wr1 = opaque(wr), ww2 = opaque(ww), wa = opaque(wr | ww);
    // A tool's own state bits change only in its own step of the sweep, so
    // the test for a task not yet known to start uses the masks as they
    // stood when the sweep began.
    const M unknown = opaque_v(~(running | done | cpu | resolved));
    // GPU tasks waiting (ready time known, not started); a task joins in its
    // own step when it is resolved there
    M waits = opaque_v(resolved & ~(running | done));
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (!((wa >> i) & 1)) continue;
      DEVMAP_KEEP_BRANCH();
      const M bi = M(1) << i;
      const uint32_t mem = opaque(tp[kHdrWords + kToolWords * i + kToolMem]);
      if ((wr1 >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        const bool on = (running >> i) & 1;
        const bool fin = on && Y[i] <= V;
        if (fin) {
          running &= ~bi;
          done |= bi;
          Y[i] = t;
        }
        const bool still = on && !fin;
        in_use = add_if(in_use, mem, still);
        vmin = still && Y[i] < vmin ? Y[i] : vmin;
      }
      if ((ww2 >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        if ((unknown >> i) & 1) {
          const M pm = load_mask<N>(tp, kHdrWords + kToolWords * i + kToolPredLo);
          if ((pm & ~(done | cpu)) == 0) {
            const uint32_t xf = tp[kHdrWords + kToolWords * i + kToolXfer];
            uint32_t r = 0;
            const M dev = DEFER && (defer & bi) ? gpu | bi : gpu;  // deferred: its GPU ready time
#pragma unroll
            for (int u = 0; u < i; ++u)
              if ((pm >> u) & 1)
                r = umax32(r, uint32_t(Y[u]) + ((((dev >> u) ^ (dev >> i)) & 1) ? xf : 0u));
            if (DEFER && (defer & bi)) {
              rgs = umin32(rgs, r);
              dhit = dhit || r <= t;
              cpu |= bi;  // parked
            } else if (gpu & bi) {
              Y[i] = r;
              resolved |= bi;
              waits |= bi;
            } else {
              const uint32_t e = r + tp[kHdrWords + kToolWords * i + kToolCpu];
              Y[i] = e;
              cpu |= bi;
              mk = umax32(mk, e);
            }
          }
        }
        if ((waits >> i) & 1) {
          const uint32_t x = uint32_t(Y[i]);
          if (x <= t) {
            if ((gqm >> i) & 1) {
              const uint32_t o = opaque(tp[kHdrWords + kToolWords * i + kToolOrig]);
              const uint64_t key = (uint64_t(x) << 32) | o;
              hk = key < hk ? key : hk;
            } else {
              starting |= bi;
              in_use += mem;
            }
          } else {
            next = umin32(next, x);  // ready later: an event, and not starting now
          }
        }
      }
    }
    if ((done | cpu) == ALL && (!DEFER || rgs == kInf)) {
      ms = umax32(t, mk);
      return true;
    }
    if (in_use > budget) return true;  // out of memory: infeasible
    // one queue admission when no queued task runs: FIFO on (ready, tool)
    if ((running & gqm) == 0 && hk != ~0ull) {
      const uint32_t head = uint32_t(hk) & kOrigLabelMask;
      if (s_mem[head] <= budget - in_use) starting |= M(1) << head;
    }
    // 4. starts, and 5. the next event: a ready time from the sweep or the
    // first GPU end at the rate of the GPU tasks now running
    running |= starting;
    uint32_t k;
    if constexpr (N <= 32) {
      k = uint32_t(__builtin_popcount(uint32_t(running)));
    } else {
      k = uint32_t(__builtin_popcountll(uint64_t(running)));
    }
    // (a task starting now was not started when the pass began)
    const M ww5 = opaque(ww);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if ((ww5 >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        if ((starting >> i) & 1) {
          Y[i] = V + (uint64_t(sh[2 * i + (((gqm >> i) & 1) ? 1 : 0)]) << 16);
          vmin = vmin < Y[i] ? vmin : Y[i];
        }
      }
    }
    uint32_t w = 0;
    if (k) {
      const uint32_t lv = (k < levels ? k : levels) - 1;
      w = sh[2 * N + lv];
      const uint64_t winv = uint64_t(sh[2 * N + levels + 2 * lv]) |
                            (uint64_t(sh[2 * N + levels + 2 * lv + 1]) << 32);
      next = umin32(next, t + uint32_t(ceil_div_small(vmin - V, w, winv)));
    }
    if (DEFER) next = umin32(next, rgs);
    if (next == kInf) return true;  // a queued task never fits
    V += uint64_t(next - t) * w;
    t = next;
    return false;
  }

  // After a DEFER prefix, with the modes now set: every parked deferred tool
  // gets the state its mode implies (its predecessors' ends are final): on
  // the CPU it ran from its ready time, on the GPU it waits from its ready
  // time.
  __host__ __device__ __forceinline__ void settle_deferred(const uint32_t* __restrict__ tab,
                                                           M defer) {
    const M gpu = gnm | gqm;
    const Tab tp = fresh(tab);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if ((defer >> i) & 1) {
        DEVMAP_KEEP_BRANCH();
        const M bi = M(1) << i;
        if (cpu & bi) {
          const M pm = load_mask<N>(tp, kHdrWords + kToolWords * i + kToolPredLo);
          const uint32_t xf = tp[kHdrWords + kToolWords * i + kToolXfer];
          uint32_t r = 0;
#pragma unroll
          for (int u = 0; u < i; ++u)
            if ((pm >> u) & 1)
              r = umax32(r, uint32_t(Y[u]) + ((((gpu >> u) ^ (gpu >> i)) & 1) ? xf : 0u));
          if (gpu & bi) {
            cpu &= ~bi;
            Y[i] = r;
            resolved |= bi;
          } else {
            const uint32_t e = r + tp[kHdrWords + kToolWords * i + kToolCpu];
            Y[i] = e;
            mk = umax32(mk, e);
          }
        }
      }
    }
  }
};

// Makespan under processor sharing, or kInf if infeasible (slot: the calling
// wave's LDS word, see wave_or).
template <int N>
__host__ __device__ __forceinline__ uint32_t evaluate_sharing(const uint32_t* __restrict__ tab,
                                                              const uint32_t* __restrict__ lds,
                                                              uint32_t levels, uint32_t budget,
                                                              MaskT<N> gnm, MaskT<N> gqm,
                                                              MaskT<N>* slot) {
  SimPS<N> sim;
  sim.init(tab, gnm, gqm);
  uint32_t ms = kInf;
  for (int pass = 0; pass < 4 * N + 4; ++pass)
    if (sim.step(tab, lds, levels, budget, pass, slot, ms)) break;
  return ms;
}

// Words [first, first + stride, ...) of the LDS image of table tab.  The
// table's duration table is label-major, dur[(2 * label + q) * levels +
// level - 1]; the image is level-major (see lds_dur_off).
template <int N>
__host__ __device__ __forceinline__ void stage_image(const uint32_t* tab, uint32_t* lds,
                                                     uint32_t first, uint32_t stride) {
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t* dur = tab + tab[kHdrDurOff];
  for (uint32_t w = first; w < uint32_t(N) * 2u * levels; w += stride) {
    const uint32_t lev = w / (2u * uint32_t(N)), iq = w - lev * (2u * uint32_t(N));
    lds[lds_dur_off<N>() + w] = dur[iq * levels + lev];
  }
  for (uint32_t i = first; i < uint32_t(N); i += stride) {
    lds[lds_mem_off<N>() + i] = tab[kHdrWords + kToolWords * i + kToolMem];
  }
}

template <int N>
__device__ __forceinline__ void stage_tables(const uint32_t* tab, uint32_t* lds) {
  stage_image<N>(tab, lds, threadIdx.x, blockDim.x);
  __syncthreads();
}

// Mode masks and index of the mapping whose enumeration positions [p0, p1)
// hold the mixed-radix digits of y (lowest first), together with the tools
// whose mode is fixed (their index contribution is the table's base).
template <int N>
__host__ __device__ __forceinline__ void decode_positions(const uint32_t* __restrict__ tab,
                                                         uint64_t y, uint32_t p0, uint32_t p1,
                                                         MaskT<N>& gn, MaskT<N>& gq,
                                                         uint64_t& x) {
  using M = MaskT<N>;
  gn = load_mask<N>(Tab{tab}, kHdrFixGnLo);
  gq = load_mask<N>(Tab{tab}, kHdrFixGqLo);
  x = uint64_t(tab[kHdrBaseLo]) | (uint64_t(tab[kHdrBaseHi]) << 32);
  for (uint32_t p = p0; p < p1; ++p) {
    const uint32_t o = tab[kEnumOptBase + p];
    const uint64_t q = opt_radix(o) == 3u ? y / 3u : y >> 1;
    const uint32_t d = uint32_t(y - uint64_t(opt_radix(o)) * q);
    const uint32_t m = opt_mode(o, d);
    const M b = M(1) << tab[kEnumLabBase + p];
    const uint64_t w = uint64_t(tab[kEnumWeightBase + 2 * p]) |
                       (uint64_t(tab[kEnumWeightBase + 2 * p + 1]) << 32);
    // (selects, not branches: a branch per mask let the optimiser pick the
    // mask through a pointer, which put both masks in scratch memory)
    gn |= m == 1u ? b : M(0);
    gq |= m == 2u ? b : M(0);
    x += uint64_t(d) * w;
    y = q;
  }
}

// Waves per SIMD the search kernel is compiled for (the register budget):
// 8 up to 19 tools, 6 beyond.  Up to 19 tools the shared-prefix LDS column
// (N words per lane) and the staged tables (sized by the problem's levels)
// let 8 blocks share a CU, and 8 waves pay for their few spilled registers.
// Measured: 19 tools 53.9 ms at 8 waves, 58.7 at 7, 64.2 at 6; random 17-
// and 18-tool DAGs 7.9 / 18.3 ms at 8 against 8.6 / 19.5 at 7.  From 20
// tools on, 64-bit indices take more registers; the 32-tool search ran 264
// ms at 6 waves against 459 at 8.
#ifndef DEVMAP_SEARCH_WAVES_SMALL
#define DEVMAP_SEARCH_WAVES_SMALL 8
#endif
#ifndef DEVMAP_SEARCH_WAVES_LARGE
#define DEVMAP_SEARCH_WAVES_LARGE 6
#endif
// The same for the processor-sharing evaluator, which keeps a 64-bit virtual
// finish per tool: 5 waves, some registers spilled (19 tools: 549 ms at 5
// waves, 594 at 4, 721 at 6; 8 waves do not fit).
#ifndef DEVMAP_SHARE_WAVES
#define DEVMAP_SHARE_WAVES 5
#endif

// Index arithmetic: 3^20 < 2^32, so up to 20 tools an index fits 32 bits.
template <int N>
using IdxT = typename std::conditional<(N <= 20), uint32_t, uint64_t>::type;

// Observer of every mapping a lane scores, called with (index, makespan or
// kInf).  Partial-range searches pass NoRecord, which compiles to nothing;
// full-range searches pass RecordTo, which writes only in a diagnostic run
// (sched_bruteforce_record); a host-side test harness records the makespans
// of a whole search through the same hook.
struct NoRecord {
  __host__ __device__ __forceinline__ bool on() const { return false; }
  __host__ __device__ __forceinline__ void operator()(uint64_t, uint32_t) const {}
};

// The search kernels' observer: writes (index, makespan) to out[index] when
// out is set (a diagnostic run), else nothing (one wave-uniform test).
struct RecordTo {
  uint32_t* out;
  __host__ __device__ __forceinline__ bool on() const { return out != nullptr; }
  __host__ __device__ __forceinline__ void operator()(uint64_t x, uint32_t ms) const {
    if (out != nullptr) out[x] = ms;
  }
};

// One lane's share of one work item: outer combination
// outer_lo + item * kBlock + lane (the digits of enumeration positions J..N-1),
// combined with every inner combination (positions 0..J-1) in range.  All
// lanes of a wave start their mappings together and step them pass by pass,
// which keeps the per-tool branches of a pass coherent across the wave.
// FULL: the whole index range in the enumeration order of the table, whose
// index need not grow along the walk, so the running minimum compares
// (makespan, index) in full.  Otherwise: index order, o * 3^J + i, clipped to
// [lo, hi); indices grow, so a strict comparison keeps the lowest index.
template <int N, bool FULL, bool SHARE, class Rec = NoRecord>
__host__ __device__ __forceinline__ void lane_search(const SearchArgs& a,
                                                     const uint32_t* __restrict__ tab,
                                                     const uint32_t* __restrict__ lds,
                                                     uint64_t item, uint32_t lane,
                                                     MaskT<N>* slot, uint32_t& best_ms,
                                                     uint64_t& best_x, Rec rec = Rec()) {
  using M = MaskT<N>;
  using I = IdxT<N>;
  const uint64_t rel = item * kBlock + lane;
  if (rel >= a.n_outer) return;
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t budget = tab[kHdrBudget];
  const uint32_t J = a.inner_digits;
  const uint64_t o = a.outer_lo + rel;
  M ogn, ogq;
  uint64_t xo64;  // index weight of the outer digits
  decode_positions<N>(tab, o, J, tab[kHdrPositions], ogn, ogq, xo64);
  uint32_t ilo = 0, ihi = a.inner_count;
  uint64_t base = 0;
  if constexpr (!FULL) {
    base = o * a.inner_count;
    const uint64_t ilo64 = a.lo > base ? a.lo - base : 0;
    const uint64_t ihi64 = a.hi - base;  // > 0 because o < ceil(hi / 3^J)
    ilo = uint32_t(ilo64 < a.inner_count ? ilo64 : a.inner_count);
    ihi = uint32_t(ihi64 < a.inner_count ? ihi64 : a.inner_count);
  }
  const I xo = I(xo64);
  I bx = I(best_x);
  // Inner digits (packed 2 bits per position), their modes and their index
  // weight: the same in every lane of the wave.  All digits start at 0.
  M ign = 0, igq = 0;
  uint32_t idig = 0;
  I xi = 0;
  for (uint32_t j = 0; j < J; ++j) {
    const uint32_t m = opt_mode(tab[kEnumOptBase + j], 0u);
    const M b = M(1) << tab[kEnumLabBase + j];
    if (m == 1u) ign |= b;
    if (m == 2u) igq |= b;
  }
  for (uint32_t i = 0; i < a.inner_count; ++i) {
    if (FULL || (i >= ilo && i < ihi)) {
      uint32_t ms;
      if constexpr (SHARE)
        ms = evaluate_sharing<N>(tab, lds, levels, budget, ogn | ign, ogq | igq, slot);
      else
        ms = evaluate<N>(tab, lds, levels, budget, ogn | ign, ogq | igq, slot);
      rec(FULL ? uint64_t(xo + xi) : base + i, ms);
      if constexpr (FULL) {
        if (ms <= best_ms) {
          const I x = xo + xi;
          if (ms < best_ms || x < bx) {
            best_ms = ms;
            bx = x;
          }
        }
      } else {
        if (ms < best_ms) {
          best_ms = ms;
          best_x = base + i;
        }
      }
    }
    // odometer step on the inner digits
    for (uint32_t j = 0; j < J; ++j) {
      const uint32_t o = tab[kEnumOptBase + j];
      const uint32_t d = (idig >> (2u * j)) & 3u;
      const M b = M(1) << tab[kEnumLabBase + j];
      const I w = I(uint64_t(tab[kEnumWeightBase + 2 * j]) |
                    (uint64_t(tab[kEnumWeightBase + 2 * j + 1]) << 32));
      ign &= ~b;
      igq &= ~b;
      const bool carry = d + 1u == opt_radix(o);
      const uint32_t m = opt_mode(o, carry ? 0u : d + 1u);
      if (m == 1u) ign |= b;
      if (m == 2u) igq |= b;
      if (!carry) {
        idig += 1u << (2u * j);
        xi += w;
        break;
      }
      idig &= ~(3u << (2u * j));
      xi -= I(d) * w;
    }
  }
  if constexpr (FULL) {
    if (best_ms != kInf) best_x = bx;
  }
}

// Shared schedule prefixes.  In a full-range search the inner (wave-uniform)
// digits are the kSharedInner tools deepest in the DAG.  Until one of them
// gets a ready time, none of them is waiting, running or resolved, so the
// schedule of the other tools, and every event time, is the same for all
// their modes: each lane runs that prefix once per outer combination, keeps
// the state it had before the first pass that resolves an inner tool, and
// restarts every inner combination from there.  With fixed-at-start
// contention an inner tool that is a sink with predecessors (the deepest
// tools are sinks) acts on no other tool before its GPU ready time, so it
// does not stop the prefix when it is resolved: the prefix runs on to the
// earliest such ready time (Sim::step<true>).  The per-tool words go to LDS
// (one column per lane), the three masks to registers.  Tools up to
// kPrefixMaxN (kPrefixMaxNShare under processor sharing).
// Every tool's word is saved and restored, inner tools included (they are
// 0): a branch per tool on the wave-uniform inner mask would be compiled as a
// lane-mask test that the compiler computes inside the prefix loop and
// reuses after it, where other lanes are active.  The exception is fixed at
// start from kCompactSnapN tools, where the search runs only with the inner
// tools on the last labels: their words are left out of the column (and read
// back as 0), a compile-time cut.
template <int N>
constexpr uint32_t snap_tools() {
  return N >= kCompactSnapN ? uint32_t(N) - kSharedInner : uint32_t(N);
}
template <int N, bool SHARE>
constexpr uint32_t snap_words() {
  // the per-tool words of the state (the masks and times stay in registers)
  return N <= (SHARE ? kPrefixMaxNShare : kPrefixMaxN)
             ? (SHARE ? uint32_t(N) + (uint32_t(N) + 1u) / 2u : snap_tools<N>())
             : 1u;
}

// A lane's saved schedule state: the per-tool words in its LDS column s, the
// rest in registers.
template <int N>
struct Snap {
  MaskT<N> started, resolved, run;
  uint32_t t, qfin, minq, mk;
};

template <int N>
__host__ __device__ __forceinline__ void snap_save(uint32_t* s, Snap<N>& m, const Sim<N>& sim) {
#pragma unroll
  for (int i = 0; i < int(snap_tools<N>()); ++i) s[i * kBlock] = sim.T[i];
  m.started = sim.started;
  m.resolved = sim.resolved;
  m.run = sim.run;
  m.t = sim.t;
  m.qfin = sim.qfin;
  m.minq = sim.minq;
  m.mk = sim.mk;
}

template <int N>
__host__ __device__ __forceinline__ void snap_load(const uint32_t* s, const Snap<N>& m,
                                                   Sim<N>& sim) {
#pragma unroll
  for (int i = 0; i < N; ++i) sim.T[i] = i < int(snap_tools<N>()) ? s[i * kBlock] : 0u;
  sim.started = m.started;
  sim.resolved = m.resolved;
  sim.run = m.run;
  sim.t = m.t;
  sim.qfin = m.qfin;
  sim.minq = m.minq;
  sim.mk = m.mk;
}

// The tools whose mode the last pass read for the first time.
template <int N>
__host__ __device__ __forceinline__ MaskT<N> first_read(const Sim<N>& sim) {
  return sim.resolved;
}

// The same for the processor-sharing evaluator: Y in LDS, 48 bits per tool
// (N low words, then the upper 16 bits of two tools per word).
template <int N>
struct SnapPS {
  MaskT<N> running, done, resolved, cpu;
  uint64_t V;
  uint32_t t, mk;
};

template <int N>
__host__ __device__ __forceinline__ void snap_save(uint32_t* s, SnapPS<N>& m,
                                                   const SimPS<N>& sim) {
  // Y < 2^47 (times below 2^30, rates at most 2^16 per us): each tool's low
  // word, then the 16 bits above it for two tools per word
#pragma unroll
  for (int i = 0; i < N; ++i) s[i * kBlock] = uint32_t(sim.Y[i]);
#pragma unroll
  for (int k = 0; 2 * k < N; ++k) {
    const uint32_t h0 = uint32_t(sim.Y[2 * k] >> 32);
    const uint32_t h1 = 2 * k + 1 < N ? uint32_t(sim.Y[2 * k + 1] >> 32) : 0u;
    s[(N + k) * kBlock] = h0 | (h1 << 16);
  }
  m.running = sim.running;
  m.done = sim.done;
  m.resolved = sim.resolved;
  m.cpu = sim.cpu;
  m.mk = sim.mk;
  m.V = sim.V;
  m.t = sim.t;
}

template <int N>
__host__ __device__ __forceinline__ void snap_load(const uint32_t* s, const SnapPS<N>& m,
                                                   SimPS<N>& sim) {
#pragma unroll
  for (int k = 0; 2 * k < N; ++k) {
    const uint32_t h = s[(N + k) * kBlock];
    sim.Y[2 * k] = uint64_t(s[(2 * k) * kBlock]) | (uint64_t(h & 0xFFFFu) << 32);
    if (2 * k + 1 < N)
      sim.Y[2 * k + 1] = uint64_t(s[(2 * k + 1) * kBlock]) | (uint64_t(h >> 16) << 32);
  }
  sim.running = m.running;
  sim.done = m.done;
  sim.resolved = m.resolved;
  sim.cpu = m.cpu;
  sim.mk = m.mk;
  sim.V = m.V;
  sim.t = m.t;
}

template <int N>
__host__ __device__ __forceinline__ MaskT<N> first_read(const SimPS<N>& sim) {
  return sim.resolved | sim.cpu;
}

// Cross-lane helpers of the shared-prefix search.  A host build has one lane
// per "wave": the ballot is the lane's own flag, its rank 0, and a pull from
// lane 0 returns the lane's own value.
__host__ __device__ __forceinline__ uint32_t lane_in_wave(uint32_t lane) {
#if defined(__HIP_DEVICE_COMPILE__)
  return lane & 63u;
#else
  (void)lane;
  return 0u;
#endif
}

// Lanes of a wave (one in a host build).
__host__ __device__ constexpr uint32_t wave_lanes() {
#if defined(__HIP_DEVICE_COMPILE__)
  return 64u;
#else
  return 1u;
#endif
}

__host__ __device__ __forceinline__ uint64_t wave_ballot(bool p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __ballot(p);
#else
  return p ? 1u : 0u;
#endif
}

// Number of lanes below the calling one whose bit is set in v.
__host__ __device__ __forceinline__ uint32_t lanes_below(uint64_t v) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_mbcnt_hi(uint32_t(v >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(v), 0u));
#else
  (void)v;
  return 0u;
#endif
}

// x of lane src (every lane of the wave must be active).
__host__ __device__ __forceinline__ uint32_t pull(uint32_t x, uint32_t src) {
#if defined(__HIP_DEVICE_COMPILE__)
  return uint32_t(__builtin_amdgcn_ds_bpermute(int(src << 2), int(x)));
#else
  (void)src;
  return x;
#endif
}

// x of this lane delivered to lane dst; dst must be a permutation of the
// wave's lanes (every lane active).
__host__ __device__ __forceinline__ uint32_t push(uint32_t x, uint32_t dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  return uint32_t(__builtin_amdgcn_ds_permute(int(dst << 2), int(x)));
#else
  (void)dst;
  return x;
#endif
}

__host__ __device__ __forceinline__ uint64_t pull64(uint64_t x, uint32_t src) {
  return uint64_t(pull(uint32_t(x), src)) | (uint64_t(pull(uint32_t(x >> 32), src)) << 32);
}

template <class M>
__host__ __device__ __forceinline__ M pull_mask(M x, uint32_t src) {
  if constexpr (sizeof(M) == 4) return pull(x, src);
  else return pull64(x, src);
}

// The register part of lane src's saved state.
template <int N>
__host__ __device__ __forceinline__ Snap<N> pull_snap(const Snap<N>& m, uint32_t src) {
  Snap<N> r;
  r.started = pull_mask(m.started, src);
  r.resolved = pull_mask(m.resolved, src);
  r.run = pull_mask(m.run, src);
  r.t = pull(m.t, src);
  r.qfin = pull(m.qfin, src);
  r.minq = pull(m.minq, src);
  r.mk = pull(m.mk, src);
  return r;
}

template <int N>
__host__ __device__ __forceinline__ SnapPS<N> pull_snap(const SnapPS<N>& m, uint32_t src) {
  SnapPS<N> r;
  r.running = pull_mask(m.running, src);
  r.done = pull_mask(m.done, src);
  r.resolved = pull_mask(m.resolved, src);
  r.cpu = pull_mask(m.cpu, src);
  r.mk = pull(m.mk, src);
  r.V = pull64(m.V, src);
  r.t = pull(m.t, src);
  return r;
}

// Full-range search with shared schedule prefixes (see above), one work item
// of a wave: the inner positions 0..kSharedInner-1 hold the deepest tools.
// SHARE: the processor-sharing evaluator, whose saved state holds Y instead
// of T.
//
// Phase 1: every lane runs the prefix of its outer combination and saves its
// state (the per-tool words in its LDS column, the rest in registers).
// Phase 2: the (prefix, inner combination) pairs of the wave's feasible
// prefixes are dealt to the lanes in rounds of 64, the inner combinations of
// one prefix in consecutive lanes: lane l of round r takes pair 64r + l, i.e.
// prefix (64r + l) / C (C inner combinations) and combination (64r + l) % C,
// restores that prefix's state from its owner (LDS column and register
// pulls) and runs the rest of the schedule.  Lanes of a round thus share few
// prefixes, so the wave-wide masks of a pass stay narrow, and lanes whose
// prefix is infeasible take no round.  Every lane of the wave must call this
// function for the same item (lanes beyond the range take part in the pulls).
template <int N, bool SHARE, class Rec = NoRecord>
__host__ __device__ __forceinline__ void lane_search_prefix(const SearchArgs& a,
                                                            const uint32_t* __restrict__ tab,
                                                            const uint32_t* __restrict__ lds,
                                                            uint64_t item, uint32_t lane,
                                                            MaskT<N>* slot, uint32_t* snap,
                                                            uint32_t& best_ms, uint64_t& best_x,
                                                            Rec rec = Rec()) {
  using M = MaskT<N>;
  using I = IdxT<N>;
  const uint64_t rel = item * kBlock + lane;
  const uint32_t wl = lane_in_wave(lane);
  uint32_t* const snap0 = snap - wl;  // LDS column of the wave's lane 0
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t budget = tab[kHdrBudget];
  constexpr uint32_t J = kSharedInner;
  static_assert(J >= 1 && J <= 2, "the pairs are dealt for one or two inner digits");
  // The inner tools (a wave-uniform mask, read through scalar loads).
  const Tab tu{tab};
  M inner = 0;
#pragma unroll
  for (uint32_t j = 0; j < J; ++j) inner |= M(1) << tu[kEnumLabBase + j];
  const M big = load_mask<N>(tu, kHdrBigLo);

  using S = typename std::conditional<SHARE, SimPS<N>, Sim<N>>::type;
  using SS = typename std::conditional<SHARE, SnapPS<N>, Snap<N>>::type;
  // (fixed at start: one pass more than a plain evaluation may take, the
  // deferred tools' GPU ready time)
  constexpr int kPasses = SHARE ? 4 * N + 4 : 2 * N + 4;
  // Inner tools that are sinks with predecessors are deferred (Sim::step):
  // the prefix runs on to their earliest GPU ready time.  The other inner
  // tools ("early") stop it before the first pass that reads one of their
  // modes, i.e. resolves one of them.  The deferred set comes from the
  // table's header, re-read where it is used rather than held in registers
  // across the rounds.
  const auto deferred = [&]() { return load_mask<N>(fresh(tab), kHdrDeferLo); };
  const M early = inner & ~load_mask<N>(tu, kHdrDeferLo);

  // Phase 1.  pstar: the pass the inner combinations restart at (-1: none,
  // the prefix is infeasible or the lane is beyond the range).
  M ogn = 0, ogq = 0;
  uint64_t xo64 = 0;
  int pstar = -1;
  SS sm{};
  if (rel < a.n_outer) {
    decode_positions<N>(tab, a.outer_lo + rel, J, tab[kHdrPositions], ogn, ogq, xo64);
    // The prefix: inner tools on the CPU (their modes are never read).
    S sim;
    sim.init(tab, ogn, ogq);
    for (int pass = 0; pass < kPasses; ++pass) {
      // (processor sharing: a deferred tool's GPU ready time can come due in
      // the pass that finds it, so that pass may have to be restarted too)
      const M defer = deferred();
      if (early || (SHARE && defer)) snap_save<N>(snap, sm, sim);
      uint32_t ms;
      const bool fin = sim.template step<true>(tab, lds, levels, budget, pass, slot, ms, defer);
      bool again = first_read<N>(sim) & early;
      if constexpr (SHARE) again = again || sim.dhit;
      if (again) {
        pstar = pass;  // restart this pass from the state saved before it
        break;
      }
      if (fin) break;  // out of memory or stuck before any inner tool: infeasible
      if (sim.t >= sim.rgs) {  // the next pass is at a deferred tool's GPU ready time
        snap_save<N>(snap, sm, sim);
        pstar = pass + 1;
        break;
      }
    }
  }

  // Phase 2: deal the (prefix, inner combination) pairs.  own: lane of the
  // rank-th feasible prefix, delivered to lane `rank` by one permutation
  // (infeasible lanes fill the lanes from nv on).
  const uint64_t feas = wave_ballot(pstar >= 0);
  const uint32_t nv = uint32_t(__builtin_popcountll(feas));
  const uint32_t rk = lanes_below(feas);
  const uint32_t owner_of_rank = push(wl, pstar >= 0 ? rk : nv + wl - rk);
  // Inner combinations: C of them, positions 0 and 1 of radices r0, r1.
  const uint32_t C = a.inner_count;
  const uint32_t o0 = tab[kEnumOptBase + 0], o1 = J > 1 ? tab[kEnumOptBase + 1] : 0u;
  const uint32_t r0 = opt_radix(o0);
  const M b0 = M(1) << tab[kEnumLabBase + 0];
  const M b1 = J > 1 ? M(1) << tab[kEnumLabBase + 1] : M(0);
  const I w0 = I(uint64_t(tab[kEnumWeightBase + 0]) | (uint64_t(tab[kEnumWeightBase + 1]) << 32));
  const I w1 = J > 1 ? I(uint64_t(tab[kEnumWeightBase + 2]) | (uint64_t(tab[kEnumWeightBase + 3]) << 32))
                     : I(0);
  const uint32_t pairs = nv * C;
  constexpr uint32_t W = wave_lanes();
  // Lane l of round r takes pair p = 64r + l = (prefix rank q, combination
  // c), q = p / C by a multiply: exact for p < 1024 and C <= 27 (the
  // multiplier's excess stays below the smallest gap to the next integer),
  // and recomputing it each round keeps no counters live across the rounds.
  const uint32_t cinv = (65536u + C - 1u) / C;
  I bx = I(best_x);
  if (rec.on() && pstar < 0 && rel < a.n_outer) {
    // an infeasible prefix: every inner combination is infeasible
    for (uint32_t cc = 0; cc < C; ++cc) {
      const uint32_t d1 = cc >= r0 ? (cc >= 2u * r0 ? 2u : 1u) : 0u;
      const uint32_t d0 = cc - d1 * r0;
      rec(uint64_t(I(xo64) + I(d0) * w0 + I(d1) * w1), kInf);
    }
  }
  for (uint32_t r0i = 0; r0i < pairs; r0i += W) {
    const uint32_t pr = r0i + wl;
    const uint32_t q = (pr * cinv) >> 16, c = pr - q * C;
    const uint32_t src = pull(owner_of_rank, q < W ? q : 0u);
    const SS ss = pull_snap<N>(sm, src);
    const M sgn = pull_mask(ogn, src), sgq = pull_mask(ogq, src);
    const I sxo = I(pull(uint32_t(xo64), src)) |
                  I(sizeof(I) > 4 ? (uint64_t(pull(uint32_t(xo64 >> 32), src)) << 32) : 0u);
    const int sps = int(pull(uint32_t(pstar), src));
    if (r0i + wl < pairs) {
      // digits of combination c: d0 = c mod r0, d1 = c div r0
      const uint32_t d1 = c >= r0 ? (c >= 2u * r0 ? 2u : 1u) : 0u;
      const uint32_t d0 = c - d1 * r0;
      const uint32_t m0 = opt_mode(o0, d0), m1 = J > 1 ? opt_mode(o1, d1) : 0u;
      S sim;
      snap_load<N>(snap0 + src, ss, sim);
      sim.gnm = sgn | (m0 == 1u ? b0 : M(0)) | (m1 == 1u ? b1 : M(0));
      sim.gqm = sgq | (m0 == 2u ? b0 : M(0)) | (m1 == 2u ? b1 : M(0));
      sim.dead = ((sim.gnm | sim.gqm) & big) != 0;
      if (const M defer = deferred()) sim.settle_deferred(tab, defer);
      const I x = sxo + I(d0) * w0 + I(d1) * w1;
      uint32_t ms = kInf;
      for (int pass = sps; pass < kPasses; ++pass)
        if (sim.step(tab, lds, levels, budget, pass, slot, ms)) break;
      rec(uint64_t(x), ms);
      if (ms <= best_ms) {
        if (ms < best_ms || x < bx) {
          best_ms = ms;
          bx = x;
        }
      }
    }
  }
  if (best_ms != kInf) best_x = bx;
}

// Exhaustive search.  Block b serves table b / blocks_per_table and walks its
// work items (kBlock consecutive outer combinations each) with a stride of
// blocks_per_table.  Each lane keeps its own (makespan, index) minimum; the
// block's minimum goes to partials[b].
template <int N, bool FULL, bool SHARE>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(
    SHARE ? (FULL && N <= kPrefixMaxNShare ? (N <= 19 ? 5 : 4)  // LDS: 1.5N words per lane
                                      : DEVMAP_SHARE_WAVES)
          : (N <= 19 ? DEVMAP_SEARCH_WAVES_SMALL
                     // from kCompactSnapN tools the shared-prefix column (N - 2 words
                     // per lane) leaves LDS for 5 blocks per CU
                     : (FULL && N >= kCompactSnapN && N <= kPrefixMaxN ? 5
                                                                        : DEVMAP_SEARCH_WAVES_LARGE))))) void
search_kernel(SearchArgs a) {
  // the staged tables: lds_words_for(N, a.lds_levels) words, sized at launch
  extern __shared__ uint32_t s_lds[];
  __shared__ uint64_t s_wave_words[kBlock / 64];  // one 8-byte word per wave
  MaskT<N>* const slot = reinterpret_cast<MaskT<N>*>(&s_wave_words[threadIdx.x / 64]);
  constexpr bool kPrefix = FULL && N <= (SHARE ? kPrefixMaxNShare : kPrefixMaxN);
  __shared__ uint32_t s_snap[kPrefix ? snap_words<N, SHARE>() * kBlock : 1];
  const uint32_t table = blockIdx.x / a.blocks_per_table;
  const uint32_t bb = blockIdx.x - table * a.blocks_per_table;
  const uint32_t* tab = a.tables + size_t(table) * a.table_stride;
  stage_tables<N>(tab, s_lds);

  uint32_t best_ms = kInf;
  uint64_t best_x = ~0ull;
  using Rec = typename std::conditional<FULL, RecordTo, NoRecord>::type;
  Rec rec{};
  if constexpr (FULL) rec.out = a.record;
  if constexpr (kPrefix) {
    if (a.prefix) {
      for (uint64_t item = bb; item < a.items_per_table; item += a.blocks_per_table)
        lane_search_prefix<N, SHARE, Rec>(a, tab, s_lds, item, threadIdx.x, slot,
                                          s_snap + threadIdx.x, best_ms, best_x, rec);
    } else {
      for (uint64_t item = bb; item < a.items_per_table; item += a.blocks_per_table)
        lane_search<N, FULL, SHARE, Rec>(a, tab, s_lds, item, threadIdx.x,
                                         slot, best_ms, best_x, rec);
    }
  } else {
    for (uint64_t item = bb; item < a.items_per_table; item += a.blocks_per_table)
      lane_search<N, FULL, SHARE, Rec>(a, tab, s_lds, item, threadIdx.x, slot,
                                       best_ms, best_x, rec);
  }

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
template <int N, bool SHARE>
__global__ __launch_bounds__(kBlock) void eval_kernel(const uint32_t* __restrict__ tab,
                                                      const uint64_t* __restrict__ idx,
                                                      int64_t n, uint64_t n_mappings,
                                                      int64_t* __restrict__ out) {
  using M = MaskT<N>;
  __shared__ uint32_t s_lds[lds_words<N>()];
  __shared__ uint64_t s_wave_words[kBlock / 64];  // one 8-byte word per wave
  MaskT<N>* const slot = reinterpret_cast<MaskT<N>*>(&s_wave_words[threadIdx.x / 64]);
  stage_tables<N>(tab, s_lds);
  const uint32_t levels = tab[kHdrLevels];
  const uint32_t budget = tab[kHdrBudget];
  for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kBlock) {
    const uint64_t x = idx[i];
    int64_t r = INT64_MAX;
    if (x < n_mappings) {
      M gn, gq;
      uint64_t xw;
      decode_positions<N>(tab, x, 0, tab[kHdrPositions], gn, gq, xw);
      uint32_t ms;
      if constexpr (SHARE)
        ms = evaluate_sharing<N>(tab, s_lds, levels, budget, gn, gq, slot);
      else
        ms = evaluate<N>(tab, s_lds, levels, budget, gn, gq, slot);
      if (ms != kInf) r = int64_t(ms);
    }
    out[i] = r;
  }
}

// Lower bound on the makespan of every mapping that gives the tools in
// `known` the modes of gn / gq (the others cpu) and leaves the rest free,
// or kInf if none of them is feasible.  Each tool lasts at least its
// shortest duration in its mode (any mode allowed to it if free) and starts
// no earlier than its predecessors end, plus its transfer when both ends
// are known to sit on different devices; the queued tools run one at a
// time, so their durations add up.
template <int N>
__host__ __device__ __forceinline__ uint32_t prefix_bound(const uint32_t* __restrict__ tab,
                                                         MaskT<N> gn, MaskT<N> gq,
                                                         MaskT<N> known) {
  using M = MaskT<N>;
  const Tab tp{tab};
  const uint32_t* bt = tab + tab[kHdrBoundOff];
  const M gpu = gn | gq;
  uint32_t C[N];
  uint32_t lb = 0, qsum = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const bool kn = (known >> i) & 1;
    const uint32_t mode = ((gn >> i) & 1) ? 1u : (((gq >> i) & 1) ? 2u : 0u);
    const uint32_t d = bt[kBoundWords * i + (kn ? mode : 3u)];
    if (d == kInf) return kInf;
    const M pm = load_mask<N>(tp, kHdrWords + kToolWords * i + kToolPredLo);
    const uint32_t xf = tp[kHdrWords + kToolWords * i + kToolXfer];
    uint32_t r = 0;
#pragma unroll
    for (int u = 0; u < i; ++u) {
      if ((pm >> u) & 1) {
        const bool cross = kn && ((known >> u) & 1) && (((gpu >> u) & 1) != ((gpu >> i) & 1));
        r = umax32(r, C[u] + (cross ? xf : 0u));
      }
    }
    C[i] = r + d;
    lb = umax32(lb, C[i]);
    if (kn && mode == 2u) qsum += d;
  }
  return umax32(lb, qsum);
}

// Bounds of prefixes [0, n): prefix y holds the mixed-radix digits of the
// table's enumeration positions [0, K); known = the labels of those tools
// and of the tools with a single allowed mode.  Prefixes whose bound does
// not exceed ub are appended to out as (bound, y) pairs; *count (zero on
// entry) receives their number.  out holds n pairs, so none is lost.
template <int N>
__global__ __launch_bounds__(kBlock) void bound_kernel(const uint32_t* __restrict__ tab,
                                                       uint32_t K, uint64_t known, int64_t n,
                                                       uint32_t ub, uint32_t* __restrict__ count,
                                                       uint2* __restrict__ out) {
  for (int64_t y = int64_t(blockIdx.x) * kBlock + threadIdx.x; y < n;
       y += int64_t(gridDim.x) * kBlock) {
    MaskT<N> gn, gq;
    uint64_t x;
    decode_positions<N>(tab, uint64_t(y), 0, K, gn, gq, x);
    const uint32_t lb = prefix_bound<N>(tab, gn, gq, MaskT<N>(known));
    if (lb != kInf && lb <= ub) {
      const uint32_t slot = atomicAdd(count, 1u);
      out[slot] = make_uint2(lb, uint32_t(y));
    }
  }
}

// Launchers of one instantiation (explicitly instantiated per tool count in
// the inst_*.hip translation units).
template <int N>
hipError_t launch_search_n(const SearchArgs& a, hipStream_t s) {
  const uint32_t blocks = a.n_tables * a.blocks_per_table;
  if (a.lds_levels < 1 || a.lds_levels > lds_levels<N>()) return hipErrorInvalidValue;
  const size_t shm = size_t(lds_words_for(N, a.lds_levels)) * 4u;
  if (a.sharing) {
    if (a.full_range)
      hipLaunchKernelGGL((search_kernel<N, true, true>), dim3(blocks), dim3(kBlock), shm, s, a);
    else
      hipLaunchKernelGGL((search_kernel<N, false, true>), dim3(blocks), dim3(kBlock), shm, s, a);
  } else {
    if (a.full_range)
      hipLaunchKernelGGL((search_kernel<N, true, false>), dim3(blocks), dim3(kBlock), shm, s, a);
    else
      hipLaunchKernelGGL((search_kernel<N, false, false>), dim3(blocks), dim3(kBlock), shm, s, a);
  }
  return hipGetLastError();
}

template <int N>
hipError_t launch_bound_n(const uint32_t* tab, uint32_t K, uint64_t known, int64_t n,
                          uint32_t ub, uint32_t* count, uint2* out, hipStream_t s) {
  int64_t blocks = (n + kBlock - 1) / kBlock;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(bound_kernel<N>, dim3(uint32_t(blocks)), dim3(kBlock), 0, s, tab, K, known,
                     n, ub, count, out);
  return hipGetLastError();
}

template <int N>
hipError_t launch_eval_n(const uint32_t* tab, const uint64_t* idx, int64_t n,
                                uint64_t n_mappings, int64_t* out, uint32_t sharing,
                                hipStream_t s) {
  int64_t blocks = (n + kBlock - 1) / kBlock;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (sharing)
    hipLaunchKernelGGL((eval_kernel<N, true>), dim3(uint32_t(blocks)), dim3(kBlock), 0, s, tab,
                       idx, n, n_mappings, out);
  else
    hipLaunchKernelGGL((eval_kernel<N, false>), dim3(uint32_t(blocks)), dim3(kBlock), 0, s, tab,
                       idx, n, n_mappings, out);
  return hipGetLastError();
}

}  // namespace devmap
