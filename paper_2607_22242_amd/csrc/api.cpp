// api.cpp -- the C ABI of include/sched_search.h: validation, topological checks,
// device problem tables, work planning, launches and result copies.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <numeric>
#include <vector>

#include "sched_search.h"
#include "devtab.h"
#include "launch.h"

using namespace devmap;

struct sched_problem {
  int32_t n = 0;
  std::vector<sched_tool> tools;
  std::vector<std::vector<int32_t>> preds;  // ascending, deduplicated
  std::vector<int32_t> order;               // order[i]: original tool with internal label i
  std::vector<int32_t> late;                // tools from the deepest in the DAG to the shallowest
  std::vector<uint32_t> contention;         // F[k-1]
  std::vector<uint8_t> allowed;             // per tool: bit m set if mode m is allowed
  std::vector<uint8_t> radix;               // number of allowed modes
  std::vector<uint64_t> weight;             // W_v: product of the radices of tools < v
  std::vector<int32_t> enum_tools;          // tools with radix > 1, ascending
  int64_t budget = 0;
  int32_t sharing = 0;                      // 1: processor-sharing contention
  bool free_fanout = false;                 // no edges, all footprints fit (kFlagFreeFanout)
  uint64_t n_mappings = 0;
  int32_t n_preds = 0;
  uint32_t table_words = 0;
  std::vector<uint32_t> table;       // device image with the problem's own latencies
  std::vector<uint32_t> table_full;  // the same, ordered for a one-table full-range search
};

namespace {

constexpr uint32_t kMaxBlocks = 65536;       // cap on search blocks per call
constexpr uint64_t kTargetLanes = 1ull << 19;  // lanes that fill an MI355X
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Mode of digit d of tool v (the d-th allowed mode, ascending).
int mode_of_digit(const sched_problem& p, int v, int d) {
  for (int m = 0; m < 3; ++m)
    if ((p.allowed[v] >> m) & 1) {
      if (d == 0) return m;
      --d;
    }
  return -1;
}

// Digit of mode m of tool v, or -1 if m is not allowed.
int digit_of_mode(const sched_problem& p, int v, int m) {
  if (m < 0 || m > 2 || !((p.allowed[v] >> m) & 1)) return -1;
  int d = 0;
  for (int k = 0; k < m; ++k) d += (p.allowed[v] >> k) & 1;
  return d;
}

// Options word of tool v's enumeration position: radix, then the mode of
// each digit.
uint32_t options_word(const sched_problem& p, int v) {
  uint32_t o = p.radix[v];
  for (int d = 0; d < p.radix[v]; ++d) o |= uint32_t(mode_of_digit(p, v, d)) << (2 + 2 * d);
  return o;
}

// round(b * f / 2^16), halves up, in 128-bit arithmetic.
uint64_t scale_q16(uint64_t b, uint32_t f) {
  unsigned __int128 p = (unsigned __int128)b * f + 32768u;
  unsigned __int128 r = p >> 16;
  return r > ~0ull ? ~0ull : uint64_t(r);
}

int check_latencies(int64_t gpu, int64_t cpu, int64_t load, int64_t xfer) {
  if (gpu < 1 || cpu < 1 || load < 0 || xfer < 0) return SCHED_E_VALUE;
  return SCHED_OK;
}

// The tools a shared-prefix search defers (header words kHdrDefer*): those
// of its inner positions 0..kSharedInner-1 that are sinks with predecessors.
// Reads the predecessor masks, the tool count and the enumeration already in
// the table.
static void write_deferred(uint32_t* table) {
  const int n = int(table[kHdrN]);
  uint64_t has_succ = 0, has_pred = 0;
  for (int i = 0; i < n; ++i) {
    const uint32_t* rec = table + kHdrWords + kToolWords * uint32_t(i);
    const uint64_t pm = uint64_t(rec[kToolPredLo]) | (uint64_t(rec[kToolPredHi]) << 32);
    has_succ |= pm;
    if (pm) has_pred |= 1ull << i;
  }
  uint64_t inner = 0;
  for (uint32_t j = 0; j < kSharedInner; ++j) inner |= 1ull << table[kEnumLabBase + j];
  const uint64_t d = inner & ~has_succ & has_pred;
  table[kHdrDeferLo] = uint32_t(d);
  table[kHdrDeferHi] = uint32_t(d >> 32);
}

// Fill the device table of problem p with latencies lat (nullptr: the
// problem's own).  Returns SCHED_E_OVERFLOW when the 32-bit guards fail.
int build_table(const sched_problem& p, const sched_lat* lat, uint32_t* out) {
  const int n = p.n;
  const int levels = std::min<int>(int(p.contention.size()), n);
  std::memset(out, 0, sizeof(uint32_t) * p.table_words);

  int64_t sum_mem = 0;
  for (const auto& t : p.tools) sum_mem += t.mem_mib;
  const int64_t budget = std::min<int64_t>(p.budget, sum_mem);
  // VRAM sums of up to N footprints (each clamped to budget+1) plus the
  // budget must stay below 2^32.
  if ((unsigned __int128)(n + 1) * (unsigned __int128)(budget + 1) >= ((unsigned __int128)1 << 32))
    return SCHED_E_OVERFLOW;

  std::vector<int32_t> label(n);
  for (int i = 0; i < n; ++i) label[p.order[i]] = i;
  uint64_t big = 0;
  unsigned __int128 bound = 0;  // worst-case makespan: sum of longest durations + transfers
  const uint32_t dur_off = kPredBase + ((uint32_t(p.n_preds) + 3u) & ~3u);
  uint32_t pred_cursor = 0;
  for (int i = 0; i < n; ++i) {
    const int v = p.order[i];
    const sched_tool& tl = p.tools[v];
    const int64_t gpu = lat ? lat[v].gpu_us : tl.gpu_us;
    const int64_t cpu = lat ? lat[v].cpu_us : tl.cpu_us;
    const int64_t load = lat ? lat[v].load_us : tl.load_us;
    const int64_t xfer = lat ? lat[v].xfer_us : tl.xfer_us;
    if (check_latencies(gpu, cpu, load, xfer) != SCHED_OK) return SCHED_E_VALUE;

    uint64_t longest = uint64_t(cpu);
    for (int q = 0; q < 2; ++q) {
      const uint64_t base = q == 0 ? uint64_t(gpu) : uint64_t(gpu) + uint64_t(load);
      for (int l = 0; l < levels; ++l) {
        const uint64_t d = scale_q16(base, p.contention[l]);
        longest = std::max(longest, d);
        if (d < (1ull << 31))
          out[dur_off + (uint32_t(i) * 2u + uint32_t(q)) * uint32_t(levels) + l] = uint32_t(d);
      }
    }
    bound += (unsigned __int128)longest + (unsigned __int128)uint64_t(xfer);
    if (bound >= ((unsigned __int128)1 << 30)) return SCHED_E_OVERFLOW;

    uint32_t* rec = out + kHdrWords + kToolWords * uint32_t(i);
    rec[kToolCpu] = uint32_t(cpu);
    rec[kToolMem] = uint32_t(std::min<int64_t>(tl.mem_mib, budget + 1));
    rec[kToolXfer] = uint32_t(xfer);
    std::vector<int32_t> pl;
    for (int32_t u : p.preds[v]) pl.push_back(label[u]);
    std::sort(pl.begin(), pl.end());
    uint64_t pm = 0;
    for (int32_t u : pl) pm |= 1ull << u;
    rec[kToolPredLo] = uint32_t(pm);
    rec[kToolPredHi] = uint32_t(pm >> 32);
    rec[kToolPredOff] = pred_cursor;
    rec[kToolNPred] = uint32_t(pl.size());
    rec[kToolOrig] = (uint32_t(v) << kOrigLabelBits) | uint32_t(i);
    for (int32_t u : pl) out[kPredBase + pred_cursor++] = uint32_t(u);
    out[kPosBase + v] = uint32_t(i);
    if (tl.mem_mib > budget) big |= 1ull << i;
  }
  // Index order: position k holds the k-th tool with a choice; the others
  // are fixed in the header.
  uint64_t fix_gn = 0, fix_gq = 0;
  for (int v = 0; v < n; ++v)
    if (p.radix[v] == 1) {
      const int m = mode_of_digit(p, v, 0);
      if (m == 1) fix_gn |= 1ull << label[v];
      if (m == 2) fix_gq |= 1ull << label[v];
    }
  for (size_t k = 0; k < p.enum_tools.size(); ++k) {
    const int v = p.enum_tools[k];
    out[kEnumLabBase + k] = uint32_t(label[v]);
    out[kEnumWeightBase + 2 * k] = uint32_t(p.weight[v]);
    out[kEnumWeightBase + 2 * k + 1] = uint32_t(p.weight[v] >> 32);
    out[kEnumOptBase + k] = options_word(p, v);
  }
  out[kHdrPositions] = uint32_t(p.enum_tools.size());
  out[kHdrFixGnLo] = uint32_t(fix_gn);
  out[kHdrFixGnHi] = uint32_t(fix_gn >> 32);
  out[kHdrFixGqLo] = uint32_t(fix_gq);
  out[kHdrFixGqHi] = uint32_t(fix_gq >> 32);
  out[kHdrN] = uint32_t(n);
  out[kHdrLevels] = uint32_t(levels);
  out[kHdrBudget] = uint32_t(budget);
  out[kHdrBigLo] = uint32_t(big);
  out[kHdrBigHi] = uint32_t(big >> 32);
  out[kHdrDurOff] = dur_off;
  write_deferred(out);
  // Processor-sharing table: isolated GPU latencies per label, then the
  // work rate of each contention level, round(2^32 / F) halves up.
  const uint32_t bound_off = dur_off + uint32_t(n) * 2u * uint32_t(levels);
  const uint32_t share_off = bound_off + kBoundWords * uint32_t(n);
  for (int i = 0; i < n; ++i) {
    const int v = p.order[i];
    const int64_t gpu = lat ? lat[v].gpu_us : p.tools[v].gpu_us;
    const int64_t load = lat ? lat[v].load_us : p.tools[v].load_us;
    out[share_off + 2 * uint32_t(i)] = uint32_t(gpu);
    out[share_off + 2 * uint32_t(i) + 1] = uint32_t(gpu + load);
  }
  for (int l = 0; l < levels; ++l) {
    const uint64_t f = p.contention[l];
    const uint64_t w = ((1ull << 33) + f) / (2 * f);
    out[share_off + 2 * uint32_t(n) + uint32_t(l)] = uint32_t(w);
    // floor(2^48 / w): the device divides by w through this reciprocal
    const uint64_t winv = (1ull << 48) / w;
    out[share_off + 2 * uint32_t(n) + uint32_t(levels) + 2 * uint32_t(l)] = uint32_t(winv);
    out[share_off + 2 * uint32_t(n) + uint32_t(levels) + 2 * uint32_t(l) + 1] = uint32_t(winv >> 32);
  }
  out[kHdrShareOff] = share_off;
  // Bound table: shortest durations per mode and over the allowed modes.
  // Fixed at start, a GPU task lasts one of its scaled durations; under
  // processor sharing at least its work over the fastest rate.
  for (int i = 0; i < n; ++i) {
    const int v = p.order[i];
    uint32_t best[3] = {out[kHdrWords + kToolWords * uint32_t(i) + kToolCpu], kInf, kInf};
    if (!((big >> i) & 1))
      for (int q = 0; q < 2; ++q)
        for (int l = 0; l < levels; ++l) {
          uint32_t d = out[dur_off + (uint32_t(i) * 2u + uint32_t(q)) * uint32_t(levels) + l];
          if (p.sharing) {
            const uint64_t work = uint64_t(out[share_off + 2 * uint32_t(i) + uint32_t(q)]) << 16;
            const uint64_t w = out[share_off + 2 * uint32_t(n) + uint32_t(l)];
            d = uint32_t((work + w - 1) / w);
          }
          best[1 + q] = std::min(best[1 + q], d);
        }
    uint32_t any = kInf;
    for (int m = 0; m < 3; ++m) {
      out[bound_off + kBoundWords * uint32_t(i) + m] = best[m];
      if ((p.allowed[v] >> m) & 1) any = std::min(any, best[m]);
    }
    out[bound_off + kBoundWords * uint32_t(i) + 3] = any;
  }
  out[kHdrBoundOff] = bound_off;
  out[kHdrFlags] = p.free_fanout ? kFlagFreeFanout : 0u;
  return SCHED_OK;
}

// Contention levels stored in a problem's table.
uint32_t table_levels(const sched_problem& p) {
  return uint32_t(std::min<int>(int(p.contention.size()), p.n));
}

// Relabel p so that the first kSharedInner tools with a choice in p.late
// (a shared-prefix search's inner digits) take the last labels, when no other
// tool depends on them: Kahn's algorithm over the other tools, lowest number
// first, then the inner tools in topological order among themselves.
// Otherwise p.order stays as it is.
static void label_inner_last(sched_problem& p) {
  const int n = p.n;
  std::vector<char> inner(n, 0);
  int taken = 0;
  for (int32_t v : p.late)
    if (p.radix[v] > 1 && taken < int(kSharedInner)) {
      inner[v] = 1;
      ++taken;
    }
  if (taken < int(kSharedInner)) return;
  std::vector<int32_t> indeg(n, 0);
  for (int32_t v = 0; v < n; ++v) indeg[v] = int32_t(p.preds[v].size());
  std::vector<int32_t> order;
  std::vector<char> done(n, 0);
  for (int pass = 0; pass < 2; ++pass) {  // the other tools, then the inner ones
    for (;;) {
      int32_t u = -1;
      for (int32_t v = 0; v < n && u < 0; ++v)
        if (!done[v] && indeg[v] == 0 && (inner[v] != 0) == (pass == 1)) u = v;
      if (u < 0) break;
      done[u] = 1;
      order.push_back(u);
      for (int32_t v = 0; v < n; ++v)
        for (int32_t x : p.preds[v])
          if (x == u) --indeg[v];
    }
    // a tool left after the first pass depends on an inner tool
    if (pass == 0 && int(order.size()) != n - int(kSharedInner)) return;
  }
  if (int(order.size()) == n) p.order = order;
}

// The first kSharedInner tools with a choice in p.late (a shared-prefix
// search's inner digits) hold the last labels.
static bool inner_last(const sched_problem& p) {
  int taken = 0;
  for (int32_t v : p.late) {
    if (p.radix[v] <= 1) continue;
    if (taken == int(kSharedInner)) break;
    ++taken;
    int32_t label = 0;
    while (p.order[label] != v) ++label;
    if (label < p.n - int(kSharedInner)) return false;
  }
  return taken == int(kSharedInner);
}

// Enumeration order (tools, inner positions first) of a search with J inner
// digits.  Index order (a partial range): the tools with a choice in
// ascending number, so that the walk follows the index.  A full range: the
// four tools deepest in the DAG take the positions right above the J inner
// digits, so that the lanes of a wave (consecutive outer combinations) differ
// in tools that act late in every schedule and step through their passes
// together; the other tools follow from deepest to shallowest.  Any order
// visits every mapping once.
// Full-range searches of problems the shared-prefix kernel serves use
// kSharedInner inner digits on the deepest tools (the kernel then computes
// each lane's schedule prefix once for all of their modes) and the next four
// deepest on the lanes: the plain deepest-first order.
bool prefix_plan(const sched_problem& p, uint64_t n_tables) {
  if (p.n > (p.sharing ? kPrefixMaxNShare : kPrefixMaxN) || p.enum_tools.size() < kSharedInner)
    return false;
  // from kCompactSnapN tools the kernel's LDS column leaves out the last labels
  if (p.n >= kCompactSnapN && !inner_last(p)) return false;
  if (p.free_fanout) return false;  // scored in closed form, nothing to share
  // enough lanes left to fill the GPU with kSharedInner inner digits
  const std::vector<int32_t>& v = p.late;
  uint64_t inner = 1;
  int taken = 0;
  for (int32_t t : v)
    if (p.radix[t] > 1 && taken < int(kSharedInner)) {
      inner *= p.radix[t];
      ++taken;
    }
  return (unsigned __int128)(p.n_mappings / inner) * n_tables >= kTargetLanes;
}

// A sequence of tools (an enumeration order) held without heap memory, so
// that planning a search allocates nothing.
struct Seq {
  int32_t v[kMaxTools];
  int n = 0;
  void push_back(int32_t x) { v[n++] = x; }
  int size() const { return n; }
  int32_t operator[](int k) const { return v[k]; }
};

Seq enumeration(const sched_problem& p, bool full, int J, bool prefix) {
  Seq seq;
  if (!full) {
    for (int32_t v : p.enum_tools) seq.push_back(v);
    return seq;
  }
  Seq late;
  for (int32_t v : p.late)
    if (p.radix[v] > 1) late.push_back(v);
  if (prefix) return late;
  const int P = late.size();
  const int lanes = std::min(4, P - J);
  for (int k = 0; k < J; ++k) seq.push_back(late[lanes + k]);
  for (int k = 0; k < lanes; ++k) seq.push_back(late[k]);
  for (int k = lanes + J; k < P; ++k) seq.push_back(late[k]);
  return seq;
}

// Replicas whose problems share this key share one search plan.
std::vector<uint8_t> plan_key(const sched_problem& p) {
  std::vector<uint8_t> k{uint8_t(p.n), uint8_t(p.sharing), uint8_t(p.free_fanout)};
  for (int32_t v : p.late)
    if (p.radix[v] > 1) k.push_back(p.radix[v]);
  return k;
}

uint64_t inner_count(const sched_problem& p, const Seq& seq, int J) {
  uint64_t c = 1;
  for (int k = 0; k < J; ++k) c *= p.radix[seq[k]];
  return c;
}

// Split [lo, hi) x n_tables into blocks of kBlock lanes; each lane owns one
// outer combination and enumerates the inner ones.  J grows while the lanes
// still number about kTargetLanes.
void plan_search(const sched_problem& p, uint64_t lo, uint64_t hi, uint32_t n_tables,
                 SearchArgs& a) {
  const bool full = lo == 0 && hi == p.n_mappings;
  const int P = int(p.enum_tools.size());
  const unsigned __int128 work = (unsigned __int128)(hi - lo) * n_tables;
  int J = 0;
  const bool prefix = full && prefix_plan(p, n_tables);
  if (prefix) {
    J = int(kSharedInner);
  } else {
    while (J < kMaxInnerDigits && J < P) {
      const uint64_t next = inner_count(p, enumeration(p, full, J + 1, false), J + 1);
      if ((unsigned __int128)next * kTargetLanes > work) break;
      ++J;
    }
  }
  const uint64_t inner = inner_count(p, enumeration(p, full, J, prefix), J);
  a.lo = lo;
  a.hi = hi;
  a.inner_digits = uint32_t(J);
  a.inner_count = uint32_t(inner);
  a.outer_lo = lo / inner;
  const uint64_t outer_hi = hi / inner + (hi % inner ? 1 : 0);
  a.n_outer = outer_hi - a.outer_lo;
  a.items_per_table = (a.n_outer + kBlock - 1) / kBlock;
  const uint64_t cap = std::max<uint64_t>(1, kMaxBlocks / n_tables);
  a.blocks_per_table = uint32_t(std::min<uint64_t>(a.items_per_table, cap));
  a.n_tables = n_tables;
  a.full_range = full ? 1u : 0u;
  a.sharing = uint32_t(p.sharing);
  a.prefix = prefix ? 1u : 0u;
  a.lds_levels = table_levels(p);
}

// Write the enumeration order seq[0..n) into a table built by build_table.
void set_enumeration(const sched_problem& p, const int32_t* seq, int n, uint32_t* table) {
  for (int k = 0; k < n; ++k) {
    const int v = seq[k];
    table[kEnumLabBase + k] = table[kPosBase + v];
    table[kEnumWeightBase + 2 * k] = uint32_t(p.weight[v]);
    table[kEnumWeightBase + 2 * k + 1] = uint32_t(p.weight[v] >> 32);
    table[kEnumOptBase + k] = options_word(p, v);
  }
  write_deferred(table);
}

void set_enumeration(const sched_problem& p, const Seq& seq, uint32_t* table) {
  set_enumeration(p, seq.v, seq.n, table);
}

void set_enumeration(const sched_problem& p, const std::vector<int32_t>& seq, uint32_t* table) {
  set_enumeration(p, seq.data(), int(seq.size()), table);
}

size_t partial_capacity(uint64_t n_tables) {
  return size_t(std::max<uint64_t>(n_tables, kMaxBlocks));
}

struct Layout {
  size_t tables, partials, results, total;
};

Layout layout_for(size_t table_bytes_total, size_t n_partials, size_t n_results) {
  Layout l;
  l.tables = 0;
  l.partials = align_up(table_bytes_total);
  l.results = l.partials + align_up(n_partials * sizeof(Partial));
  l.total = l.results + align_up(n_results * sizeof(DevResult));
  return l;
}

int check_workspace(void* ws, size_t ws_bytes, size_t need) {
  if (ws == nullptr) return SCHED_E_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return SCHED_E_WORKSPACE;
  if (ws_bytes < need) return SCHED_E_WORKSPACE;
  return SCHED_OK;
}

#define HIP_TRY(expr)                                  \
  do {                                                 \
    if ((expr) != hipSuccess) return SCHED_E_DEVICE;   \
  } while (0)

int create_problem(const sched_tool* tools, int32_t n_tools, const sched_edge* edges,
                   int32_t n_edges, const uint32_t* contention_q16, int32_t n_levels,
                   int64_t vram_budget_mib, const uint8_t* allowed, int32_t sharing,
                   sched_problem** out) {
  if (out == nullptr || tools == nullptr || contention_q16 == nullptr) return SCHED_E_NULL;
  if (n_edges > 0 && edges == nullptr) return SCHED_E_NULL;
  if (n_tools < 1 || n_tools > kMaxTools || n_edges < 0 || n_levels < 1 || n_levels > kMaxLevels)
    return SCHED_E_SIZE;
  if (vram_budget_mib < 0) return SCHED_E_VALUE;
  for (int32_t v = 0; v < n_tools; ++v) {
    const sched_tool& t = tools[v];
    if (check_latencies(t.gpu_us, t.cpu_us, t.load_us, t.xfer_us) != SCHED_OK || t.mem_mib < 0)
      return SCHED_E_VALUE;
  }
  for (int32_t l = 0; l < n_levels; ++l)
    if (contention_q16[l] < 65536u || contention_q16[l] > (1u << 24)) return SCHED_E_VALUE;
  if (allowed != nullptr)
    for (int32_t v = 0; v < n_tools; ++v)
      if (allowed[v] < 1 || allowed[v] > 7) return SCHED_E_VALUE;
  if (sharing != 0 && sharing != 1) return SCHED_E_VALUE;

  sched_problem* p = new (std::nothrow) sched_problem;
  if (p == nullptr) return SCHED_E_NOMEM;
  try {
    p->n = n_tools;
    p->sharing = sharing;
    p->tools.assign(tools, tools + n_tools);
    p->contention.assign(contention_q16, contention_q16 + n_levels);
    p->budget = vram_budget_mib;
    p->preds.assign(n_tools, {});
    for (int32_t e = 0; e < n_edges; ++e) {
      const int32_t u = edges[e].src, v = edges[e].dst;
      if (u < 0 || u >= n_tools || v < 0 || v >= n_tools || u == v) {
        delete p;
        return SCHED_E_EDGE;
      }
      p->preds[v].push_back(u);
    }
    int32_t total = 0;
    for (auto& pl : p->preds) {
      std::sort(pl.begin(), pl.end());
      pl.erase(std::unique(pl.begin(), pl.end()), pl.end());
      total += int32_t(pl.size());
    }
    p->n_preds = total;
    // Kahn's algorithm: every tool must be reachable in a topological order.
    std::vector<int32_t> indeg(n_tools, 0);
    std::vector<std::vector<int32_t>> succ(n_tools);
    for (int32_t v = 0; v < n_tools; ++v)
      for (int32_t u : p->preds[v]) {
        succ[u].push_back(v);
        indeg[v]++;
      }
    // Kahn's algorithm, always taking the lowest-numbered ready tool: the
    // internal labels of the device tables (a cycle leaves tools unlabelled).
    std::vector<char> done(n_tools, 0);
    for (int32_t step = 0; step < n_tools; ++step) {
      int32_t u = -1;
      for (int32_t v = 0; v < n_tools && u < 0; ++v)
        if (!done[v] && indeg[v] == 0) u = v;
      if (u < 0) break;
      done[u] = 1;
      p->order.push_back(u);
      for (int32_t v : succ[u]) --indeg[v];
    }
    if (int32_t(p->order.size()) != n_tools) {
      delete p;
      return SCHED_E_CYCLE;
    }
    // Depth of every tool (longest chain from a source, in tools) and its
    // number of ancestors, in topological order; deepest first, ties to
    // more ancestors, then to the lower tool number.
    std::vector<int32_t> depth(n_tools, 1);
    std::vector<std::vector<char>> anc(n_tools, std::vector<char>(n_tools, 0));
    for (int32_t v : p->order)
      for (int32_t u : p->preds[v]) {
        depth[v] = std::max(depth[v], depth[u] + 1);
        anc[v][u] = 1;
        for (int32_t w = 0; w < n_tools; ++w)
          if (anc[u][w]) anc[v][w] = 1;
      }
    std::vector<int32_t> n_anc(n_tools, 0);
    for (int32_t v = 0; v < n_tools; ++v)
      for (int32_t w = 0; w < n_tools; ++w) n_anc[v] += anc[v][w];
    p->late.resize(n_tools);
    std::iota(p->late.begin(), p->late.end(), 0);
    std::stable_sort(p->late.begin(), p->late.end(), [&](int32_t a, int32_t b) {
      if (depth[a] != depth[b]) return depth[a] > depth[b];
      return n_anc[a] > n_anc[b];
    });
    // Decision space: allowed modes, radices and mixed-radix weights.
    p->allowed.assign(n_tools, uint8_t(7));
    if (allowed != nullptr) p->allowed.assign(allowed, allowed + n_tools);
    p->radix.resize(n_tools);
    p->weight.resize(n_tools);
    uint64_t w = 1;
    for (int32_t v = 0; v < n_tools; ++v) {
      const uint8_t a = p->allowed[v];
      p->radix[v] = uint8_t((a & 1) + ((a >> 1) & 1) + ((a >> 2) & 1));
      p->weight[v] = w;
      w *= p->radix[v];
      if (p->radix[v] > 1) p->enum_tools.push_back(v);
    }
    p->n_mappings = w;
    int64_t sum_mem = 0;
    for (const sched_tool& t : p->tools) sum_mem += t.mem_mib;
    const bool fanout_fits = total == 0 && sharing == 0 && p->budget >= sum_mem;
    if (n_tools >= kCompactSnapN && n_tools <= kPrefixMaxN && sharing == 0 && !fanout_fits)
      label_inner_last(*p);
    bool identity = true;
    for (int32_t i = 0; i < n_tools; ++i) identity = identity && p->order[i] == i;
    p->free_fanout = fanout_fits && identity;
    p->table_words = table_words(n_tools, total, std::min<int>(n_levels, n_tools));
    p->table.assign(p->table_words, 0u);
    const int rc = build_table(*p, nullptr, p->table.data());
    if (rc != SCHED_OK) {
      delete p;
      return rc;
    }
    // the table of a one-table full-range search, in its enumeration order
    SearchArgs a{};
    plan_search(*p, 0, p->n_mappings, 1, a);
    p->table_full = p->table;
    set_enumeration(*p, enumeration(*p, true, int(a.inner_digits), a.prefix != 0),
                    p->table_full.data());
  } catch (const std::bad_alloc&) {
    delete p;
    return SCHED_E_NOMEM;
  }
  *out = p;
  return SCHED_OK;
}

// One what-if candidate around a base mapping.
struct Cand {
  int kind, tool, mode, swap_tool;  // kind 0 base, 1 single-tool move, 2 swap
};

// The base mapping and its neighbourhood in the order of Algorithm 1: for
// each tool i and each other allowed mode a, the move i -> a, followed, when
// a is gpu_now, by one swap per tool j on gpu_now that may use gpu_queue
// (i -> gpu_now, j -> gpu_queue).  Every swap is listed; callers decide
// which to keep.
void neighbourhood(const sched_problem& p, uint64_t base, std::vector<uint64_t>& idx,
                   std::vector<Cand>& cands) {
  const int n = p.n;
  std::vector<int32_t> d(n);
  sched_mapping_modes(&p, base, d.data());
  // Moving tool v from mode d[v] to mode a changes its digit, weighted by W_v.
  auto with = [&](uint64_t x, int v, int a) {
    return x - uint64_t(digit_of_mode(p, v, d[v])) * p.weight[v] +
           uint64_t(digit_of_mode(p, v, a)) * p.weight[v];
  };
  auto ok = [&](int v, int a) { return ((p.allowed[v] >> a) & 1) != 0; };
  idx.clear();
  cands.clear();
  idx.push_back(base);
  cands.push_back({0, -1, -1, -1});
  for (int i = 0; i < n; ++i)
    for (int a = 0; a < 3; ++a) {
      if (a == d[i] || !ok(i, a)) continue;
      idx.push_back(with(base, i, a));
      cands.push_back({1, i, a, -1});
      if (a == 1)
        for (int j = 0; j < n; ++j)
          if (j != i && d[j] == 1 && ok(j, 2)) {
            idx.push_back(with(with(base, i, 1), j, 2));
            cands.push_back({2, i, 1, j});
          }
    }
}

// ---------------------------------------------------------------------------
// Exact search with pruning.

constexpr uint64_t kPruneMinSpace = 1ull << 22;  // smaller spaces: one exhaustive search
constexpr uint64_t kMaxPrefixes = 1ull << 24;    // bounded prefix assignments per call
constexpr uint64_t kMinSubspace = 1ull << 12;    // mappings per searched subspace, at least
constexpr uint32_t kChunkTables = 2048;          // subspaces per search launch

// The prefix: tools with a choice whose shortest durations differ most
// between their modes come first (their choice moves the bound most), then
// as many as fit kMaxPrefixes while the subspaces keep kMinSubspace mappings.
struct PrunePlan {
  std::vector<int32_t> prefix;  // prefix tools, digit order of the prefix index
  uint64_t n_prefixes = 1;
  uint64_t subspace = 1;        // mappings per prefix
};

PrunePlan plan_prune(const sched_problem& p) {
  PrunePlan pl;
  const uint32_t* bt = p.table.data() + p.table[kHdrBoundOff];
  std::vector<std::pair<uint64_t, int32_t>> spread;
  for (int32_t v : p.enum_tools) {
    const uint32_t i = p.table[kPosBase + v];
    uint32_t lo = kInf, hi = 0;
    for (int m = 0; m < 3; ++m) {
      if (!((p.allowed[v] >> m) & 1)) continue;
      const uint32_t d = bt[kBoundWords * i + m];
      lo = std::min(lo, d);
      hi = std::max(hi, d == kInf ? (1u << 30) : d);
    }
    spread.push_back({uint64_t(hi - lo), v});
  }
  std::stable_sort(spread.begin(), spread.end(),
                   [](const auto& a, const auto& b) { return a.first > b.first; });
  pl.subspace = p.n_mappings;
  for (const auto& sv : spread) {
    const uint64_t r = p.radix[sv.second];
    if (pl.n_prefixes * r > kMaxPrefixes || pl.subspace / r < kMinSubspace) break;
    pl.prefix.push_back(sv.second);
    pl.n_prefixes *= r;
    pl.subspace /= r;
  }
  return pl;
}

struct PruneLayout {
  size_t tables, partials, results, bounds, probe_idx, probe_ms, total;
};

PruneLayout prune_layout(const sched_problem& p, const PrunePlan& pl) {
  PruneLayout l;
  const size_t probes = size_t(1 + 2 * p.n + p.n * (p.n - 1));
  l.tables = 0;
  l.partials = align_up(size_t(kChunkTables) * p.table_words * 4);
  l.results = l.partials + align_up(partial_capacity(kChunkTables) * sizeof(Partial));
  l.bounds = l.results + align_up(size_t(kChunkTables) * sizeof(DevResult));
  // Survivor count (one word, padded) and then up to n_prefixes (bound, y)
  // pairs.
  l.probe_idx = l.bounds + align_up(4) + align_up(size_t(pl.n_prefixes) * 8);
  l.probe_ms = l.probe_idx + align_up(probes * 8);
  l.total = l.probe_ms + align_up(probes * 8);
  return l;
}

// Workspace bytes of one search over one problem table.
size_t one_search_bytes(const sched_problem& p) {
  return layout_for(size_t(p.table_words) * 4, partial_capacity(1), 1).total;
}

// One search of [lo, hi) in workspace ws (at least one_search_bytes): table
// copy, search and reduction on stream s, then the result.  record: every
// mapping's makespan (full ranges only; null: none).  Allocates nothing.
int search_one(const sched_problem& p, uint64_t lo, uint64_t hi, char* ws, hipStream_t s,
               uint32_t* record, sched_result* h_out) {
  const Layout L = layout_for(size_t(p.table_words) * 4, partial_capacity(1), 1);
  SearchArgs a{};
  plan_search(p, lo, hi, 1, a);
  a.tables = reinterpret_cast<const uint32_t*>(ws + L.tables);
  a.table_stride = p.table_words;
  a.partials = reinterpret_cast<Partial*>(ws + L.partials);
  a.record = record;
  DevResult* d_res = reinterpret_cast<DevResult*>(ws + L.results);
  const std::vector<uint32_t>& table = a.full_range ? p.table_full : p.table;
  HIP_TRY(hipMemcpyAsync(ws + L.tables, table.data(), size_t(p.table_words) * 4,
                         hipMemcpyHostToDevice, s));
  HIP_TRY(launch_search(p.n, a, s));
  HIP_TRY(launch_reduce(a.partials, a.blocks_per_table, 1, d_res, s));
  DevResult r;
  HIP_TRY(hipMemcpyAsync(&r, d_res, sizeof(r), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  h_out->best_index = r.index;
  h_out->makespan_us = r.makespan;
  return SCHED_OK;
}

}  // namespace

extern "C" {

int sched_problem_create(const sched_tool* tools, int32_t n_tools, const sched_edge* edges,
                         int32_t n_edges, const uint32_t* contention_q16, int32_t n_levels,
                         int64_t vram_budget_mib, sched_problem** out) {
  return create_problem(tools, n_tools, edges, n_edges, contention_q16, n_levels,
                        vram_budget_mib, nullptr, 0, out);
}

int sched_problem_create_desc(const sched_problem_desc* d, sched_problem** out) {
  if (d == nullptr) return SCHED_E_NULL;
  return create_problem(d->tools, d->n_tools, d->edges, d->n_edges, d->contention_q16,
                        d->n_levels, d->vram_budget_mib, d->allowed, d->contention_mode, out);
}

int sched_problem_create_masked(const sched_tool* tools, int32_t n_tools,
                                const sched_edge* edges, int32_t n_edges,
                                const uint32_t* contention_q16, int32_t n_levels,
                                int64_t vram_budget_mib, const uint8_t* allowed,
                                sched_problem** out) {
  if (allowed == nullptr) return SCHED_E_NULL;
  return create_problem(tools, n_tools, edges, n_edges, contention_q16, n_levels,
                        vram_budget_mib, allowed, 0, out);
}

void sched_problem_destroy(sched_problem* p) { delete p; }

int sched_mapping_modes(const sched_problem* p, uint64_t index, int32_t* modes) {
  if (p == nullptr || modes == nullptr) return SCHED_E_NULL;
  if (index >= p->n_mappings) return SCHED_E_RANGE;
  for (int v = 0; v < p->n; ++v) {
    const int d = int(index % p->radix[v]);
    index /= p->radix[v];
    modes[v] = mode_of_digit(*p, v, d);
  }
  return SCHED_OK;
}

int sched_mapping_index(const sched_problem* p, const int32_t* modes, uint64_t* index) {
  if (p == nullptr || modes == nullptr || index == nullptr) return SCHED_E_NULL;
  uint64_t x = 0;
  for (int v = 0; v < p->n; ++v) {
    const int d = digit_of_mode(*p, v, modes[v]);
    if (d < 0) return SCHED_E_VALUE;
    x += uint64_t(d) * p->weight[v];
  }
  *index = x;
  return SCHED_OK;
}

int sched_num_tools(const sched_problem* p, int32_t* out) {
  if (p == nullptr || out == nullptr) return SCHED_E_NULL;
  *out = p->n;
  return SCHED_OK;
}

int sched_num_mappings(const sched_problem* p, uint64_t* out) {
  if (p == nullptr || out == nullptr) return SCHED_E_NULL;
  *out = p->n_mappings;
  return SCHED_OK;
}

int sched_workspace_bytes(const sched_problem* const* problems, int32_t n_problems,
                          int32_t n_replicas, size_t* out) {
  if (problems == nullptr || out == nullptr) return SCHED_E_NULL;
  if (n_problems < 1 || n_replicas < 0) return SCHED_E_SIZE;
  size_t max_stride = 0;
  for (int32_t i = 0; i < n_problems; ++i) {
    if (problems[i] == nullptr) return SCHED_E_NULL;
    max_stride = std::max<size_t>(max_stride, problems[i]->table_words);
  }
  // single-problem calls
  size_t need = layout_for(max_stride * 4, partial_capacity(1), 1).total;
  if (n_replicas > 0) {
    const size_t r = size_t(n_replicas);
    need = std::max(need, layout_for(r * max_stride * 4, partial_capacity(r), r).total);
  }
  *out = need;
  return SCHED_OK;
}

int sched_bruteforce_argmin(const sched_problem* p, uint64_t lo, uint64_t hi, void* d_workspace,
                            size_t ws_bytes, void* hip_stream, sched_result* h_out) {
  if (p == nullptr || h_out == nullptr) return SCHED_E_NULL;
  if (lo >= hi || hi > p->n_mappings) return SCHED_E_RANGE;
  const int rc = check_workspace(d_workspace, ws_bytes, one_search_bytes(*p));
  if (rc != SCHED_OK) return rc;
  return search_one(*p, lo, hi, static_cast<char*>(d_workspace),
                    reinterpret_cast<hipStream_t>(hip_stream), nullptr, h_out);
}

int sched_bruteforce_argmin_noalloc(const sched_problem* p, uint64_t lo, uint64_t hi,
                                    void* hip_stream, sched_result* h_out) {
  if (p == nullptr || h_out == nullptr) return SCHED_E_NULL;
  if (lo >= hi || hi > p->n_mappings) return SCHED_E_RANGE;
  if (one_search_bytes(*p) > kScratchBytes) return SCHED_E_WORKSPACE;
  void* ws = nullptr;
  HIP_TRY(scratch_buffer(&ws));
  return search_one(*p, lo, hi, static_cast<char*>(ws), reinterpret_cast<hipStream_t>(hip_stream),
                    nullptr, h_out);
}

int sched_bruteforce_record(const sched_problem* p, void* d_workspace, size_t ws_bytes,
                            void* hip_stream, uint32_t* d_makespan, uint64_t capacity,
                            sched_result* h_out) {
  if (p == nullptr || h_out == nullptr || d_makespan == nullptr) return SCHED_E_NULL;
  if (capacity < p->n_mappings) return SCHED_E_WORKSPACE;
  const int rc = check_workspace(d_workspace, ws_bytes, one_search_bytes(*p));
  if (rc != SCHED_OK) return rc;
  return search_one(*p, 0, p->n_mappings, static_cast<char*>(d_workspace),
                    reinterpret_cast<hipStream_t>(hip_stream), d_makespan, h_out);
}

int sched_eval_batch(const sched_problem* const* problems, int32_t n_problems,
                     const int32_t* replica_problem, const sched_lat* replica_lat,
                     int32_t n_replicas, void* d_workspace, size_t ws_bytes, void* hip_stream,
                     sched_result* h_out) {
  if (problems == nullptr || replica_problem == nullptr || replica_lat == nullptr ||
      h_out == nullptr)
    return SCHED_E_NULL;
  if (n_problems < 1 || n_replicas < 1) return SCHED_E_SIZE;
  size_t max_stride = 0;
  for (int32_t i = 0; i < n_problems; ++i) {
    if (problems[i] == nullptr) return SCHED_E_NULL;
    max_stride = std::max<size_t>(max_stride, problems[i]->table_words);
  }
  std::vector<size_t> lat_off(static_cast<size_t>(n_replicas));
  size_t off = 0;
  for (int32_t r = 0; r < n_replicas; ++r) {
    const int32_t pi = replica_problem[r];
    if (pi < 0 || pi >= n_problems) return SCHED_E_RANGE;
    lat_off[r] = off;
    off += size_t(problems[pi]->n);
  }
  const size_t R = size_t(n_replicas);
  const Layout L = layout_for(R * max_stride * 4, partial_capacity(R), R);
  int rc = check_workspace(d_workspace, ws_bytes, L.total);
  if (rc != SCHED_OK) return rc;

  // Replicas grouped by search plan: tool count (one kernel instantiation
  // per count) and the radices along the enumeration order, which fix the
  // inner digits and the outer combinations.
  std::vector<std::vector<uint8_t>> keys(static_cast<size_t>(n_problems));
  for (int32_t i = 0; i < n_problems; ++i) keys[size_t(i)] = plan_key(*problems[i]);
  std::vector<int32_t> order(R);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
    return keys[size_t(replica_problem[x])] < keys[size_t(replica_problem[y])];
  });
  std::vector<uint32_t> host_tables;
  std::vector<DevResult> host_res;
  try {
    host_tables.assign(R * max_stride, 0u);
    host_res.resize(R);
  } catch (const std::bad_alloc&) {
    return SCHED_E_NOMEM;
  }
  // Per group of equal tool count: the search plan, then the tables.
  struct Group {
    size_t first, last;
    SearchArgs a;
  };
  std::vector<Group> groups;
  for (size_t first = 0; first < R;) {
    const int32_t pf = replica_problem[order[first]];
    size_t last = first;
    while (last < R && keys[size_t(replica_problem[order[last]])] == keys[size_t(pf)]) ++last;
    Group g{first, last, SearchArgs{}};
    const sched_problem& p0 = *problems[pf];
    plan_search(p0, 0, p0.n_mappings, uint32_t(last - first), g.a);
    for (size_t i = first; i < last; ++i)
      g.a.lds_levels = std::max(g.a.lds_levels, table_levels(*problems[replica_problem[order[i]]]));
    // The block cap is shared by the whole batch so partials stay bounded.
    const uint64_t cap = std::max<uint64_t>(1, kMaxBlocks / R);
    g.a.blocks_per_table = uint32_t(std::min<uint64_t>(g.a.items_per_table, cap));
    groups.push_back(g);
    first = last;
  }
  for (const Group& g : groups) {
    for (size_t i = g.first; i < g.last; ++i) {
      const int32_t r = order[i];
      const sched_problem& p = *problems[replica_problem[r]];
      uint32_t* tb = host_tables.data() + i * max_stride;
      rc = build_table(p, replica_lat + lat_off[r], tb);
      if (rc != SCHED_OK) return rc;
      set_enumeration(p, enumeration(p, true, int(g.a.inner_digits), g.a.prefix != 0), tb);
    }
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  char* ws = static_cast<char*>(d_workspace);
  const uint32_t* d_tables = reinterpret_cast<const uint32_t*>(ws + L.tables);
  Partial* d_partials = reinterpret_cast<Partial*>(ws + L.partials);
  DevResult* d_res = reinterpret_cast<DevResult*>(ws + L.results);
  HIP_TRY(hipMemcpyAsync(ws + L.tables, host_tables.data(), R * max_stride * 4,
                         hipMemcpyHostToDevice, s));
  size_t partial_cursor = 0;
  for (Group& g : groups) {
    const int n = problems[replica_problem[order[g.first]]]->n;
    const uint32_t count = uint32_t(g.last - g.first);
    SearchArgs& a = g.a;
    a.tables = d_tables + g.first * max_stride;
    a.table_stride = uint32_t(max_stride);
    a.partials = d_partials + partial_cursor;
    HIP_TRY(launch_search(n, a, s));
    HIP_TRY(launch_reduce(a.partials, a.blocks_per_table, count, d_res + g.first, s));
    partial_cursor += size_t(count) * a.blocks_per_table;
  }
  HIP_TRY(hipMemcpyAsync(host_res.data(), d_res, R * sizeof(DevResult), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  for (size_t i = 0; i < R; ++i) {
    h_out[order[i]].best_index = host_res[i].index;
    h_out[order[i]].makespan_us = host_res[i].makespan;
  }
  return SCHED_OK;
}

int sched_eval_mappings_device(const sched_problem* p, const uint64_t* d_idx, int64_t n,
                               int64_t* d_makespan, void* d_workspace, size_t ws_bytes,
                               void* hip_stream) {
  if (p == nullptr) return SCHED_E_NULL;
  if (n < 0) return SCHED_E_SIZE;
  if (n == 0) return SCHED_OK;
  if (d_idx == nullptr || d_makespan == nullptr) return SCHED_E_NULL;
  const size_t need = align_up(size_t(p->table_words) * 4);
  int rc = check_workspace(d_workspace, ws_bytes, need);
  if (rc != SCHED_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  HIP_TRY(hipMemcpyAsync(d_workspace, p->table.data(), size_t(p->table_words) * 4,
                         hipMemcpyHostToDevice, s));
  HIP_TRY(launch_eval(p->n, static_cast<const uint32_t*>(d_workspace), d_idx, n, p->n_mappings,
                      d_makespan, uint32_t(p->sharing), s));
  HIP_TRY(hipStreamSynchronize(s));
  return SCHED_OK;
}

int sched_eval_mappings(const sched_problem* p, const uint64_t* h_idx, int64_t n,
                        void* d_workspace, size_t ws_bytes, void* hip_stream,
                        int64_t* h_makespan) {
  if (p == nullptr) return SCHED_E_NULL;
  if (n < 0) return SCHED_E_SIZE;
  if (n == 0) return SCHED_OK;
  if (h_idx == nullptr || h_makespan == nullptr) return SCHED_E_NULL;
  for (int64_t i = 0; i < n; ++i)
    if (h_idx[i] >= p->n_mappings) return SCHED_E_RANGE;
  // the table, then chunks of indices and makespans (8 bytes each) in the
  // rest of the workspace
  const size_t head = align_up(size_t(p->table_words) * 4);
  int rc = check_workspace(d_workspace, ws_bytes, head + kAlign + 16);
  if (rc != SCHED_OK) return rc;
  // chunk indices, then chunk makespans at the next 256-byte boundary: fits
  const int64_t chunk = int64_t(std::min<size_t>((ws_bytes - head - kAlign) / 16, size_t(1) << 24));
  char* ws = static_cast<char*>(d_workspace);
  uint64_t* d_idx = reinterpret_cast<uint64_t*>(ws + head);
  int64_t* d_out = reinterpret_cast<int64_t*>(ws + head + align_up(size_t(chunk) * 8));
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  HIP_TRY(hipMemcpyAsync(ws, p->table.data(), size_t(p->table_words) * 4,
                         hipMemcpyHostToDevice, s));
  for (int64_t at = 0; at < n; at += chunk) {
    const int64_t m = std::min(chunk, n - at);
    HIP_TRY(hipMemcpyAsync(d_idx, h_idx + at, size_t(m) * 8, hipMemcpyHostToDevice, s));
    HIP_TRY(launch_eval(p->n, reinterpret_cast<const uint32_t*>(ws), d_idx, m, p->n_mappings,
                        d_out, uint32_t(p->sharing), s));
    HIP_TRY(hipMemcpyAsync(h_makespan + at, d_out, size_t(m) * 8, hipMemcpyDeviceToHost, s));
  }
  HIP_TRY(hipStreamSynchronize(s));
  return SCHED_OK;
}

int sched_eval_reprobes(const sched_problem* p, uint64_t base_index, const sched_lat* lat,
                        void* d_workspace, size_t ws_bytes, void* hip_stream,
                        sched_probe* h_out, int32_t capacity, int32_t* n_out) {
  if (p == nullptr || h_out == nullptr || n_out == nullptr) return SCHED_E_NULL;
  if (base_index >= p->n_mappings) return SCHED_E_RANGE;
  const int n = p->n;
  const int64_t worst = 1 + 2 * int64_t(n) + int64_t(n) * (n - 1);
  if (capacity < worst) return SCHED_E_SIZE;
  const Layout L = layout_for(size_t(p->table_words) * 4, partial_capacity(1), 1);
  int rc = check_workspace(d_workspace, ws_bytes, L.total);
  if (rc != SCHED_OK) return rc;

  std::vector<uint32_t> table;
  std::vector<uint64_t> idx;
  std::vector<int64_t> ms;
  try {
    table.assign(p->table_words, 0u);
    idx.reserve(size_t(worst));
  } catch (const std::bad_alloc&) {
    return SCHED_E_NOMEM;
  }
  if (lat != nullptr) {
    rc = build_table(*p, lat, table.data());
    if (rc != SCHED_OK) return rc;
  } else {
    table = p->table;
  }
  std::vector<Cand> cands;
  try {
    neighbourhood(*p, base_index, idx, cands);
  } catch (const std::bad_alloc&) {
    return SCHED_E_NOMEM;
  }
  const size_t m = idx.size();
  ms.assign(m, 0);
  // Scratch for the index list and the makespans: the partials region.
  if (m * 16 > partial_capacity(1) * sizeof(Partial)) return SCHED_E_WORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  char* ws = static_cast<char*>(d_workspace);
  uint64_t* d_idx = reinterpret_cast<uint64_t*>(ws + L.partials);
  int64_t* d_ms = reinterpret_cast<int64_t*>(ws + L.partials + m * 8);
  HIP_TRY(hipMemcpyAsync(ws + L.tables, table.data(), size_t(p->table_words) * 4,
                         hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(d_idx, idx.data(), m * 8, hipMemcpyHostToDevice, s));
  HIP_TRY(launch_eval(n, reinterpret_cast<const uint32_t*>(ws + L.tables), d_idx, int64_t(m),
                      p->n_mappings, d_ms, uint32_t(p->sharing), s));
  HIP_TRY(hipMemcpyAsync(ms.data(), d_ms, m * 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  // Keep a swap only when its move to gpu_now was infeasible.
  int32_t out = 0;
  int64_t move_ms = 0;
  for (size_t k = 0; k < m; ++k) {
    const Cand& c = cands[k];
    if (c.kind == 1) move_ms = ms[k];
    if (c.kind == 2 && move_ms != INT64_MAX) continue;
    sched_probe& pr = h_out[out++];
    pr.index = idx[k];
    pr.makespan_us = ms[k];
    pr.kind = c.kind;
    pr.tool = c.tool;
    pr.mode = c.mode;
    pr.swap_tool = c.swap_tool;
  }
  *n_out = out;
  return SCHED_OK;
}

int sched_pruned_workspace_bytes(const sched_problem* p, size_t* out) {
  if (p == nullptr || out == nullptr) return SCHED_E_NULL;
  const size_t plain = layout_for(size_t(p->table_words) * 4, partial_capacity(1), 1).total;
  size_t need = plain;
  if (p->n_mappings >= kPruneMinSpace) need = std::max(need, prune_layout(*p, plan_prune(*p)).total);
  *out = need;
  return SCHED_OK;
}

int sched_pruned_argmin(const sched_problem* p, void* d_workspace, size_t ws_bytes,
                        void* hip_stream, sched_result* h_out, sched_prune_stats* stats) {
  if (p == nullptr || h_out == nullptr) return SCHED_E_NULL;
  sched_prune_stats st{};
  if (p->n_mappings < kPruneMinSpace) {  // not worth bounding: one exhaustive search
    const int rc = sched_bruteforce_argmin(p, 0, p->n_mappings, d_workspace, ws_bytes, hip_stream,
                                           h_out);
    if (rc == SCHED_OK && stats != nullptr) {
      st.prefixes = 1;
      st.prefixes_searched = 1;
      st.mappings_searched = p->n_mappings;
      st.launches = 1;
      st.shared_prefix_launches = prefix_plan(*p, 1) ? 1 : 0;
      st.initial_bound_us = INT64_MAX;
      *stats = st;
    }
    return rc;
  }
  const int n = p->n;
  const PrunePlan pl = plan_prune(*p);
  const PruneLayout L = prune_layout(*p, pl);
  int rc = check_workspace(d_workspace, ws_bytes, L.total);
  if (rc != SCHED_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  char* ws = static_cast<char*>(d_workspace);
  const uint32_t* d_tab = reinterpret_cast<const uint32_t*>(ws + L.tables);
  const uint32_t stride = p->table_words;

  try {
    // 1. Upper bound: steepest descent over the what-if neighbourhood of
    // Algorithm 1 (every single-tool move and swap), from index 0.
    uint64_t ub_x = 0;
    int64_t ub_ms = INT64_MAX;
    {
      std::vector<uint64_t> idx;
      std::vector<Cand> cands;
      std::vector<int64_t> ms;
      HIP_TRY(hipMemcpyAsync(ws + L.tables, p->table.data(), size_t(stride) * 4,
                             hipMemcpyHostToDevice, s));
      uint64_t x = 0;
      for (int round = 0; round < 4 * n + 4; ++round) {
        neighbourhood(*p, x, idx, cands);
        ms.assign(idx.size(), 0);
        uint64_t* d_idx = reinterpret_cast<uint64_t*>(ws + L.probe_idx);
        int64_t* d_ms = reinterpret_cast<int64_t*>(ws + L.probe_ms);
        HIP_TRY(hipMemcpyAsync(d_idx, idx.data(), idx.size() * 8, hipMemcpyHostToDevice, s));
        HIP_TRY(launch_eval(n, d_tab, d_idx, int64_t(idx.size()), p->n_mappings, d_ms,
                            uint32_t(p->sharing), s));
        HIP_TRY(hipMemcpyAsync(ms.data(), d_ms, idx.size() * 8, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        ++st.descent_rounds;
        size_t best = 0;
        for (size_t k = 1; k < idx.size(); ++k)
          if (ms[k] < ms[best] || (ms[k] == ms[best] && idx[k] < idx[best])) best = k;
        if (ms[best] < ub_ms || (ms[best] == ub_ms && idx[best] < ub_x)) {
          ub_ms = ms[best];
          ub_x = idx[best];
        }
        if (best == 0) break;  // no neighbour improves on x
        x = idx[best];
      }
    }
    st.initial_bound_us = ub_ms;

    // 2. Bounds of every prefix assignment.
    std::vector<uint32_t> btab(p->table);
    std::vector<int32_t> seq(pl.prefix);
    for (int32_t v : p->enum_tools)
      if (std::find(pl.prefix.begin(), pl.prefix.end(), v) == pl.prefix.end()) seq.push_back(v);
    set_enumeration(*p, seq, btab.data());
    uint64_t known = 0;
    for (int32_t v : pl.prefix) known |= 1ull << p->table[kPosBase + v];
    for (int v = 0; v < n; ++v)
      if (p->radix[v] == 1) known |= 1ull << p->table[kPosBase + v];
    HIP_TRY(hipMemcpyAsync(ws + L.tables, btab.data(), size_t(stride) * 4, hipMemcpyHostToDevice,
                           s));
    uint32_t* d_count = reinterpret_cast<uint32_t*>(ws + L.bounds);
    uint2* d_live = reinterpret_cast<uint2*>(ws + L.bounds + align_up(4));
    const uint32_t ub32 = ub_ms == INT64_MAX ? kInf - 1 : uint32_t(ub_ms);
    HIP_TRY(hipMemsetAsync(d_count, 0, 4, s));
    HIP_TRY(launch_bound(n, d_tab, uint32_t(pl.prefix.size()), known, int64_t(pl.n_prefixes), ub32,
                         d_count, d_live, s));
    uint32_t n_live = 0;
    HIP_TRY(hipMemcpyAsync(&n_live, d_count, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (n_live > pl.n_prefixes) return SCHED_E_DEVICE;
    std::vector<uint2> raw(n_live);
    if (n_live) {
      HIP_TRY(hipMemcpyAsync(raw.data(), d_live, size_t(n_live) * 8, hipMemcpyDeviceToHost, s));
      HIP_TRY(hipStreamSynchronize(s));
    }
    st.prefixes = pl.n_prefixes;
    st.prefix_tools = int32_t(pl.prefix.size());

    // Survivors: bound <= upper bound (equal bounds may hide a lower index),
    // most promising first; the kernel appends them in no fixed order.
    std::vector<std::pair<uint32_t, uint64_t>> live(n_live);
    for (uint32_t i = 0; i < n_live; ++i) live[i] = {raw[i].x, raw[i].y};
    std::sort(live.begin(), live.end());

    // 3. Subspaces: the prefix tools fixed, the rest enumerated with the
    // weights of the full index.
    sched_problem sub = *p;
    for (int32_t v : pl.prefix) sub.allowed[v] = uint8_t(1u << mode_of_digit(*p, v, 0));
    sub.enum_tools.clear();
    sub.n_mappings = 1;
    for (int v = 0; v < n; ++v) {
      const uint8_t a = sub.allowed[v];
      sub.radix[v] = uint8_t((a & 1) + ((a >> 1) & 1) + ((a >> 2) & 1));
      if (sub.radix[v] > 1) sub.enum_tools.push_back(v);
      sub.n_mappings *= sub.radix[v];
    }
    std::vector<uint32_t> stab(stride);
    rc = build_table(sub, nullptr, stab.data());
    if (rc != SCHED_OK) return rc;
    const uint64_t fix_gn0 = uint64_t(p->table[kHdrFixGnLo]) | (uint64_t(p->table[kHdrFixGnHi]) << 32);
    const uint64_t fix_gq0 = uint64_t(p->table[kHdrFixGqLo]) | (uint64_t(p->table[kHdrFixGqHi]) << 32);

    uint64_t best_x = ub_ms == INT64_MAX ? ~0ull : ub_x;
    int64_t best_ms = ub_ms;
    std::vector<uint32_t> tables;
    std::vector<DevResult> res;
    size_t next = 0;
    while (next < live.size()) {
      if (best_ms != INT64_MAX && int64_t(live[next].first) > best_ms) break;
      size_t end = next;
      while (end < live.size() && end - next < kChunkTables &&
             (best_ms == INT64_MAX || int64_t(live[end].first) <= best_ms))
        ++end;
      const uint32_t count = uint32_t(end - next);
      SearchArgs a{};
      plan_search(sub, 0, sub.n_mappings, count, a);
      set_enumeration(sub, enumeration(sub, true, int(a.inner_digits), a.prefix != 0), stab.data());
      tables.assign(size_t(count) * stride, 0u);
      for (uint32_t t = 0; t < count; ++t) {
        uint32_t* tb = tables.data() + size_t(t) * stride;
        std::copy(stab.begin(), stab.end(), tb);
        uint64_t y = live[next + t].second, base = 0, gn = fix_gn0, gq = fix_gq0;
        for (int32_t v : pl.prefix) {
          const int d = int(y % p->radix[v]);
          y /= p->radix[v];
          base += uint64_t(d) * p->weight[v];
          const int m = mode_of_digit(*p, v, d);
          const uint64_t b = 1ull << p->table[kPosBase + v];
          if (m == 1) gn |= b;
          if (m == 2) gq |= b;
        }
        tb[kHdrFixGnLo] = uint32_t(gn);
        tb[kHdrFixGnHi] = uint32_t(gn >> 32);
        tb[kHdrFixGqLo] = uint32_t(gq);
        tb[kHdrFixGqHi] = uint32_t(gq >> 32);
        tb[kHdrBaseLo] = uint32_t(base);
        tb[kHdrBaseHi] = uint32_t(base >> 32);
      }
      a.tables = d_tab;
      a.table_stride = stride;
      a.partials = reinterpret_cast<Partial*>(ws + L.partials);
      DevResult* d_res = reinterpret_cast<DevResult*>(ws + L.results);
      HIP_TRY(hipMemcpyAsync(ws + L.tables, tables.data(), tables.size() * 4,
                             hipMemcpyHostToDevice, s));
      HIP_TRY(launch_search(n, a, s));
      HIP_TRY(launch_reduce(a.partials, a.blocks_per_table, count, d_res, s));
      res.resize(count);
      HIP_TRY(hipMemcpyAsync(res.data(), d_res, count * sizeof(DevResult), hipMemcpyDeviceToHost,
                             s));
      HIP_TRY(hipStreamSynchronize(s));
      for (const DevResult& r : res)
        if (r.makespan < best_ms || (r.makespan == best_ms && r.index < best_x)) {
          best_ms = r.makespan;
          best_x = r.index;
        }
      st.prefixes_searched += count;
      st.mappings_searched += uint64_t(count) * sub.n_mappings;
      st.launches += 1;
      st.shared_prefix_launches += a.prefix ? 1 : 0;
      next = end;
    }
    h_out->best_index = best_ms == INT64_MAX ? ~0ull : best_x;
    h_out->makespan_us = best_ms;
  } catch (const std::bad_alloc&) {
    return SCHED_E_NOMEM;
  }
  if (stats != nullptr) *stats = st;
  return SCHED_OK;
}

int sched_valu_probe(uint32_t blocks, uint32_t iters, uint32_t* d_out, void* hip_stream,
                     double* lane_ops) {
  if (d_out == nullptr || lane_ops == nullptr) return SCHED_E_NULL;
  if (blocks == 0 || iters == 0 || blocks > (1u << 24)) return SCHED_E_SIZE;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  double ops = 0;
  HIP_TRY(launch_valu_probe(blocks, iters, d_out, s, &ops));
  HIP_TRY(hipStreamSynchronize(s));
  *lane_ops = ops;
  return SCHED_OK;
}

int sched_wave_or_probe(const uint64_t* d_in, const uint8_t* d_active, uint32_t blocks,
                        uint64_t* d_out64, uint32_t* d_out32, void* hip_stream) {
  if (d_in == nullptr || d_active == nullptr || d_out64 == nullptr || d_out32 == nullptr)
    return SCHED_E_NULL;
  if (blocks == 0 || blocks > (1u << 16)) return SCHED_E_SIZE;
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  HIP_TRY(launch_wave_or_probe(d_in, d_active, blocks, d_out64, d_out32, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SCHED_OK;
}

const char* sched_strerror(int code) {
  switch (code) {
    case SCHED_OK: return "ok";
    case SCHED_E_NULL: return "null pointer argument";
    case SCHED_E_SIZE: return "size out of range";
    case SCHED_E_VALUE: return "value out of range";
    case SCHED_E_EDGE: return "edge endpoint out of range or self-loop";
    case SCHED_E_CYCLE: return "edges contain a cycle";
    case SCHED_E_RANGE: return "index range or replica map out of range";
    case SCHED_E_OVERFLOW: return "times or VRAM sums would not fit the 32-bit device path";
    case SCHED_E_WORKSPACE: return "workspace null, misaligned or too small";
    case SCHED_E_DEVICE: return "HIP runtime error";
    case SCHED_E_NOMEM: return "host allocation failed";
    default: return "unknown error";
  }
}

}  // extern "C"
