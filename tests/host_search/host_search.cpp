// host_search.cpp -- test harness: the search kernels' per-lane code
// (lane_search_prefix / lane_search from kernels.h) compiled for the host
// and driven over every work item of a full-range search plan, one lane per
// "wave" (the wave-wide ORs reduce to the lane's own masks).  The problem
// tables, enumeration order and plan come from the library's own host code
// (api.cpp, included here); device launches are stubbed out.  Prints the
// lowest-(makespan, index) mapping: "<index> <makespan> <prefix 0|1>".
// With a second argument, also writes every mapping's makespan (uint32 per
// index, 0xFFFFFFFF infeasible) to that file ("-" for none); a third argument
// "share" selects the processor-sharing reading of contention.
//
// Input (text, argv[1], "-" for stdin): n_tools n_edges n_levels budget,
// then n_tools lines "gpu cpu load xfer mem", n_edges lines "src dst", then
// the n_levels Q16 contention factors.
#include "../../paper_2607_22242_amd/csrc/api.cpp"
#include "../../paper_2607_22242_amd/csrc/kernels.h"

#include <cstdio>
#include <vector>

namespace devmap {
hipError_t launch_search(int, const SearchArgs&, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_eval(int, const uint32_t*, const uint64_t*, int64_t, uint64_t, int64_t*,
                       uint32_t, hipStream_t) {
  return hipErrorUnknown;
}
hipError_t launch_bound(int, const uint32_t*, uint32_t, uint64_t, int64_t, uint32_t, uint32_t*,
                        uint2*, hipStream_t) {
  return hipErrorUnknown;
}
hipError_t launch_reduce(const Partial*, uint32_t, uint32_t, DevResult*, hipStream_t) {
  return hipErrorUnknown;
}
hipError_t launch_valu_probe(uint32_t, uint32_t, uint32_t*, hipStream_t, double*) {
  return hipErrorUnknown;
}
hipError_t launch_wave_or_probe(const uint64_t*, const uint8_t*, uint32_t, uint64_t*, uint32_t*,
                                hipStream_t) {
  return hipErrorUnknown;
}
hipError_t scratch_buffer(void**) { return hipErrorUnknown; }
}  // namespace devmap

using namespace devmap;

// Stores each scored mapping's makespan at its index.
struct Table {
  uint32_t* ms;
  bool on() const { return true; }
  void operator()(uint64_t x, uint32_t m) const { ms[x] = m; }
};

template <int N, bool SHARE>
static void run(const sched_problem* p, const char* table_path) {
  // unwritten entries keep a value no makespan or infeasible mark takes
  std::vector<uint32_t> all(table_path ? p->n_mappings : 0, 0xFFFFFFFEu);
  const Table rec{all.data()};
  SearchArgs a{};
  plan_search(*p, 0, p->n_mappings, 1, a);
  std::vector<uint32_t> table = p->table;
  set_enumeration(*p, enumeration(*p, true, int(a.inner_digits), a.prefix != 0), table.data());
  const uint32_t* tab = table.data();
  // the block's LDS image (stage_tables)
  std::vector<uint32_t> lds(lds_words_for(N, tab[kHdrLevels]));
  stage_image<N>(tab, lds.data(), 0, 1);
  uint32_t gms = kInf;
  uint64_t gx = ~0ull;
#pragma omp parallel
  {
    std::vector<uint32_t> snap(snap_words<N, SHARE>() * kBlock);
    uint64_t slot_word = 0;
    MaskT<N>* slot = reinterpret_cast<MaskT<N>*>(&slot_word);
    uint32_t bms = kInf;
    uint64_t bx = ~0ull;
#pragma omp for schedule(dynamic, 16)
    for (long long item = 0; item < (long long)a.items_per_table; ++item) {
      for (uint32_t lane = 0; lane < uint32_t(kBlock); ++lane) {
        uint32_t ms = kInf;
        uint64_t x = ~0ull;
        if (a.prefix && table_path)
          lane_search_prefix<N, SHARE, Table>(a, tab, lds.data(), uint64_t(item), lane, slot,
                                              snap.data() + lane, ms, x, rec);
        else if (a.prefix)
          lane_search_prefix<N, SHARE>(a, tab, lds.data(), uint64_t(item), lane, slot,
                                       snap.data() + lane, ms, x);
        else if (table_path)
          lane_search<N, true, SHARE, Table>(a, tab, lds.data(), uint64_t(item), lane, slot,
                                             ms, x, rec);
        else
          lane_search<N, true, SHARE>(a, tab, lds.data(), uint64_t(item), lane, slot, ms, x);
        if (ms < bms || (ms == bms && x < bx)) {
          bms = ms;
          bx = x;
        }
      }
    }
#pragma omp critical
    {
      if (bms < gms || (bms == gms && bx < gx)) {
        gms = bms;
        gx = bx;
      }
    }
  }
  printf("%llu %u %u\n", (unsigned long long)gx, gms, a.prefix);
  if (table_path) {
    FILE* out = fopen(table_path, "wb");
    if (!out || fwrite(all.data(), 4, all.size(), out) != all.size()) {
      printf("error writing %s\n", table_path);
    }
    if (out) fclose(out);
  }
}

int main(int argc, char** argv) {
  FILE* f = (argc > 1 && argv[1][0] != '-') ? fopen(argv[1], "r") : stdin;
  const char* table_path = argc > 2 && argv[2][0] != '-' ? argv[2] : nullptr;
  const bool share = argc > 3 && argv[3][0] == 's';
  if (!f) return 2;
  int n, ne, nl;
  long long budget;
  if (fscanf(f, "%d %d %d %lld", &n, &ne, &nl, &budget) != 4) return 2;
  std::vector<sched_tool> tools(n);
  for (auto& t : tools) {
    long long g, c, l, x, m;
    if (fscanf(f, "%lld %lld %lld %lld %lld", &g, &c, &l, &x, &m) != 5) return 2;
    t = sched_tool{g, c, l, x, m};
  }
  std::vector<sched_edge> e(ne);
  for (auto& x : e)
    if (fscanf(f, "%d %d", &x.src, &x.dst) != 2) return 2;
  std::vector<uint32_t> F(nl);
  for (auto& x : F)
    if (fscanf(f, "%u", &x) != 1) return 2;
  sched_problem* p = nullptr;
  sched_problem_desc desc{tools.data(), n, e.data(), ne, F.data(), nl, budget, nullptr,
                          share ? 1 : 0};
  const int rc = sched_problem_create_desc(&desc, &p);
  if (rc != SCHED_OK) {
    printf("error %d\n", rc);
    return 1;
  }
#ifdef HOST_SEARCH_ONLY_N
  // a build for one tool count (the sanitizer build, which is slow to compile)
  if (n != HOST_SEARCH_ONLY_N) {
    printf("error tools\n");
    return 1;
  }
  if (share)
    run<HOST_SEARCH_ONLY_N, true>(p, table_path);
  else
    run<HOST_SEARCH_ONLY_N, false>(p, table_path);
#else
  switch (n) {
// (the processor-sharing lanes are built for 14 tools only, to keep the
// harness quick to compile)
#define HOST_SEARCH_CASE(K)                      \
  case K:                                        \
    if (!share)                                  \
      run<K, false>(p, table_path);              \
    else if constexpr (K == 14)                  \
      run<K, true>(p, table_path);               \
    else                                         \
      printf("error tools\n");                   \
    break;
    HOST_SEARCH_CASE(6) HOST_SEARCH_CASE(7) HOST_SEARCH_CASE(8) HOST_SEARCH_CASE(9)
    HOST_SEARCH_CASE(10) HOST_SEARCH_CASE(11) HOST_SEARCH_CASE(12) HOST_SEARCH_CASE(13)
    HOST_SEARCH_CASE(14) HOST_SEARCH_CASE(15) HOST_SEARCH_CASE(16)
    default:
      printf("error tools\n");
      return 1;
  }
#endif
  sched_problem_destroy(p);
  return 0;
}
