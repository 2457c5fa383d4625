// monitor.cpp -- sliding-window latency statistics of the runtime monitor's
// observation feedback (Section 3.2, Algorithm 1, passive path), and the
// re-measured latencies they give for re-scoring.  Host-only.
#include <algorithm>
#include <deque>
#include <new>
#include <vector>

#include "sched_search.h"

struct sched_monitor {
  int32_t n = 0;
  int32_t window = 0;
  std::vector<std::deque<int64_t>> obs;  // [tool * 3 + mode]: the newest `window` latencies
};

namespace {

// Mean of a window, rounded half up (all values are non-negative).
int64_t window_mean(const std::deque<int64_t>& w) {
  __int128 sum = 0;
  for (int64_t x : w) sum += x;
  const __int128 c = __int128(w.size());
  return int64_t((2 * sum + c) / (2 * c));
}

}  // namespace

extern "C" {

int sched_monitor_create(int32_t n_tools, int32_t window, sched_monitor** out) {
  if (out == nullptr) return SCHED_E_NULL;
  if (n_tools < 1 || n_tools > 40 || window < 1) return SCHED_E_SIZE;
  sched_monitor* m = new (std::nothrow) sched_monitor;
  if (m == nullptr) return SCHED_E_NOMEM;
  try {
    m->n = n_tools;
    m->window = window;
    m->obs.resize(size_t(n_tools) * 3);
  } catch (const std::bad_alloc&) {
    delete m;
    return SCHED_E_NOMEM;
  }
  *out = m;
  return SCHED_OK;
}

void sched_monitor_destroy(sched_monitor* m) { delete m; }

int sched_monitor_observe(sched_monitor* m, const int32_t* modes, const int64_t* latency_us) {
  if (m == nullptr || modes == nullptr || latency_us == nullptr) return SCHED_E_NULL;
  for (int32_t v = 0; v < m->n; ++v)
    if (modes[v] < 0 || modes[v] > 2) return SCHED_E_VALUE;
  try {
    for (int32_t v = 0; v < m->n; ++v) {
      if (latency_us[v] < 0) continue;  // not observed this round
      std::deque<int64_t>& w = m->obs[size_t(v) * 3 + size_t(modes[v])];
      w.push_back(latency_us[v]);
      if (int32_t(w.size()) > m->window) w.pop_front();
    }
  } catch (const std::bad_alloc&) {
    return SCHED_E_NOMEM;
  }
  return SCHED_OK;
}

int sched_monitor_averages(const sched_monitor* m, int64_t* mean_us, int32_t* count) {
  if (m == nullptr || mean_us == nullptr || count == nullptr) return SCHED_E_NULL;
  for (size_t k = 0; k < m->obs.size(); ++k) {
    count[k] = int32_t(m->obs[k].size());
    mean_us[k] = m->obs[k].empty() ? 0 : window_mean(m->obs[k]);
  }
  return SCHED_OK;
}

int sched_monitor_latencies(const sched_monitor* m, const sched_tool* profile, sched_lat* out) {
  if (m == nullptr || profile == nullptr || out == nullptr) return SCHED_E_NULL;
  for (int32_t v = 0; v < m->n; ++v) {
    const std::deque<int64_t>& wc = m->obs[size_t(v) * 3 + 0];
    const std::deque<int64_t>& wn = m->obs[size_t(v) * 3 + 1];
    const std::deque<int64_t>& wq = m->obs[size_t(v) * 3 + 2];
    sched_lat l;
    l.cpu_us = wc.empty() ? profile[v].cpu_us : std::max<int64_t>(1, window_mean(wc));
    l.gpu_us = wn.empty() ? profile[v].gpu_us : std::max<int64_t>(1, window_mean(wn));
    l.load_us = wq.empty() ? profile[v].load_us : std::max<int64_t>(0, window_mean(wq) - l.gpu_us);
    l.xfer_us = profile[v].xfer_us;
    out[v] = l;
  }
  return SCHED_OK;
}

}  // extern "C"
