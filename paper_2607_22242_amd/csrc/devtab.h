// devtab.h -- device-side problem table and launch arguments (internal).
//
// One table per problem (or per replica in a batch) is a flat array of
// 32-bit words, written by the host into the caller's workspace and read by
// the kernels with uniform (scalar) loads, except the duration table which
// each block stages in LDS because its index depends on the lane.
//
// Tools are stored under internal labels 0..N-1 that follow a topological
// order of the DAG (every predecessor has a smaller label), so one ascending
// sweep over the labels sees each tool after all of its predecessors.  The
// mapping index keeps the caller's tool numbering: it is mixed radix, digit v
// being the rank of original tool v's mode among the r_v modes allowed to it
// (r_v = 3 when all are), with weight W_v = r_0 r_1 ... r_(v-1).  Tools with a
// single allowed mode take no digit: their mode is fixed in the header.
#pragma once
#include <stdint.h>

namespace devmap {

constexpr int kMaxTools = 40;
constexpr int kMaxLevels = 64;
constexpr uint32_t kInf = 0xFFFFFFFFu;  // "never": unknown ready time, infeasible
constexpr int kBlock = 256;             // threads per search block (4 waves)
constexpr int kMaxInnerDigits = 6;      // inner (wave-uniform) digits per lane
#ifndef DEVMAP_SHARED_INNER
#define DEVMAP_SHARED_INNER 2
#endif
constexpr uint32_t kSharedInner = DEVMAP_SHARED_INNER;  // inner digits of a shared-prefix search
constexpr int kPrefixMaxN = 32;         // tool counts served by shared prefixes (fixed at start:
                                        // N LDS words per lane)
constexpr int kPrefixMaxNShare = 24;    // the same under processor sharing (1.5N words per lane)
// From this many tools a fixed-at-start shared-prefix search needs its inner
// tools on the last kSharedInner labels: their words (0 whenever a prefix
// saves its state) are left out of the LDS column, so that N - kSharedInner
// words per lane leave room for 5 blocks per CU up to kPrefixMaxN tools.
constexpr int kCompactSnapN = 27;
static_assert(kCompactSnapN > kPrefixMaxNShare, "the compact column is fixed-at-start only");

// Header words.
enum : uint32_t {
  kHdrN = 0,          // number of tools
  kHdrLevels = 1,     // contention levels stored = min(K, N)
  kHdrBudget = 2,     // VRAM budget, clamped to the summed footprint
  kHdrBigLo = 3,      // tools whose footprint exceeds the budget (bits 0..31)
  kHdrBigHi = 4,      //                                           (bits 32..63)
  kHdrDurOff = 5,     // word offset of the duration table
  kHdrPositions = 6,  // P: tools with more than one allowed mode (digit positions)
  kHdrFixGnLo = 7,    // labels of tools fixed on gpu_now (bits 0..31)
  kHdrFixGnHi = 8,    //                                   (bits 32..63)
  kHdrFixGqLo = 9,    // labels of tools fixed on gpu_queue
  kHdrFixGqHi = 10,
  kHdrBaseLo = 11,    // index contribution of the fixed tools (a subspace's
  kHdrBaseHi = 12,    // offset in the mapping index)
  kHdrBoundOff = 13,  // word offset of the bound table
  kHdrShareOff = 14,  // word offset of the processor-sharing table
  kHdrFlags = 15,     // kFlag* bits
  kHdrDeferLo = 16,   // inner tools of a shared-prefix search that are sinks with
  kHdrDeferHi = 17,   // predecessors: the search defers them (bits 0..31, 32..63)
  kHdrWords = 18,
};

// A fan-out (no edges) whose footprints all fit the budget together, scored
// with fixed-at-start contention: every tool is ready at 0, no start can run
// out of memory and no queued tool waits for VRAM, so a mapping's schedule
// follows in closed form (evaluate_fanout).  Its internal labels are the
// original tool numbers.
constexpr uint32_t kFlagFreeFanout = 1u;

// Record of the tool with internal label i at kHdrWords + kToolWords * i.
enum : uint32_t {
  kToolCpu = 0,       // cpu_us
  kToolMem = 1,       // footprint, clamped to budget + 1
  kToolXfer = 2,      // input transfer across devices
  kToolPredLo = 3,    // predecessor mask bits 0..31
  kToolPredHi = 4,    // predecessor mask bits 32..63
  kToolPredOff = 5,   // offset of the predecessor list (from kPredBase)
  kToolNPred = 6,     // number of predecessors
  kToolOrig = 7,      // (original tool number << kOrigLabelBits) | label
  kToolWords = 8,
};

// kToolOrig holds the original number above the label, so that the lowest
// word among candidate tools names both the first in the queue's tie order and
// its label.
constexpr uint32_t kOrigLabelBits = 6;
constexpr uint32_t kOrigLabelMask = (1u << kOrigLabelBits) - 1u;
static_assert(kMaxTools <= (1 << kOrigLabelBits), "labels must fit below the original number");

// pos[v]: internal label of original tool v.
constexpr uint32_t kPosBase = kHdrWords + kToolWords * kMaxTools;  // 338
// Enumeration order of a search over positions 0..P-1: position p holds the
// digit of the tool with internal label elab[p], whose weight in the mapping
// index is ew[p] = W_v of its original number v (two words, low first), and
// whose options eo[p] give its radix (bits 0-1, 2 or 3) and the mode of
// digit d in bits 2+2d..3+2d.  Positions 0..J-1 are the inner digits, J.. the
// outer ones.
constexpr uint32_t kEnumLabBase = kPosBase + kMaxTools;          // 378
constexpr uint32_t kEnumWeightBase = kEnumLabBase + kMaxTools;   // 418
constexpr uint32_t kEnumOptBase = kEnumWeightBase + 2 * kMaxTools;  // 498
// Predecessor lists (internal labels), then the duration table.
constexpr uint32_t kPredBase = kEnumOptBase + kMaxTools;  // 538

// Radix and digit -> mode of an enumeration position's options word.
inline constexpr uint32_t opt_radix(uint32_t o) { return o & 3u; }
inline constexpr uint32_t opt_mode(uint32_t o, uint32_t d) { return (o >> (2u + 2u * d)) & 3u; }

// Duration table: dur[(i * 2 + q) * levels + (level - 1)] for internal label
// i, q = 0 for gpu_now (base gpu_us), q = 1 for gpu_queue (gpu_us + load_us).
//
// Bound table (after the duration table): for internal label i, four words
// bt[4i + m] = the shortest duration tool i can have in mode m (cpu, gpu_now,
// gpu_queue: the least over contention levels), and bt[4i + 3] = the least
// of those over the modes the problem allows it; kInf for a GPU mode of a
// tool whose footprint exceeds the budget (it can never run there).
constexpr uint32_t kBoundWords = 4;

// Processor-sharing table (after the bound table): for internal label i,
// b[2i] = gpu_us and b[2i + 1] = gpu_us + load_us (isolated latencies), then
// for each contention level the work rate w = round(2^32 / F) in 2^-16 us of
// isolated work per us, then for each level floor(2^48 / w) (two words, low
// first), the reciprocal the device divides by.
inline uint32_t table_words(int n, int n_preds, int levels) {
  uint32_t dur_off = kPredBase + ((uint32_t(n_preds) + 3u) & ~3u);
  return dur_off + uint32_t(n) * 2u * uint32_t(levels) + kBoundWords * uint32_t(n) +
         2u * uint32_t(n) + 3u * uint32_t(levels);
}

struct Partial {
  uint64_t index;
  uint32_t makespan;
  uint32_t pad;
};

struct SearchArgs {
  const uint32_t* tables;     // n_tables tables, table_stride words apart
  Partial* partials;          // one per block
  uint64_t lo, hi;            // index range searched in every table
  uint64_t outer_lo;          // first outer combination
  uint64_t n_outer;           // outer combinations covering [lo, hi)
  uint32_t table_stride;
  uint32_t n_tables;
  uint32_t inner_digits;      // J: enumeration positions 0..J-1 are walked per lane
  uint32_t inner_count;       // product of the radices of positions 0..J-1
  uint64_t items_per_table;   // ceil(n_outer / kBlock)
  uint32_t blocks_per_table;
  uint32_t full_range;        // 1: [lo, hi) is every mapping, any enumeration order
  uint32_t sharing;           // 1: processor-sharing contention
  uint32_t prefix;            // 1: shared prefixes (kSharedInner inner digits on the
                              //    deepest tools, full range, fixed at start)
  uint32_t lds_levels;        // the most contention levels any of the tables stores
  uint32_t* record;           // full range, one table: every scored mapping's makespan
                              // (kInf if infeasible) goes to record[index]; null: none
};

struct DevResult {
  uint64_t index;
  int64_t makespan;
};

}  // namespace devmap
