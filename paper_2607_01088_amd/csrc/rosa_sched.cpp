// Profiling-guided System-1 batch-size selection (host only): the closed-loop
// worker simulation and the choice of include/rosa_sched.h.
#include <algorithm>
#include <cmath>
#include <vector>

#include "../../include/rosa_sched.h"

namespace {

// Value of rank ceil(num / den * n) (1-based) of sorted values.
double rank_value(const std::vector<double> &sorted, long num, long den) {
  const long n = (long)sorted.size();
  long r = (num * n + den - 1) / den;
  r = std::max(1L, std::min(n, r));
  return sorted[r - 1];
}

void simulate(int robots, int b, double batch_ms, double t_act_ms, int n_batches, rosa_s1_outcome &o) {
  o = rosa_s1_outcome{};
  o.batch = b;
  if (robots < b) return;                 // a batch of b never fills
  o.feasible = 1;
  std::vector<double> submit(robots, 0.0);   // time of each robot's pending request
  std::vector<int> order(robots);
  std::vector<double> lat;
  lat.reserve((size_t)b * (n_batches - n_batches / 2));
  const int warm = n_batches / 2;
  double free_at = 0.0, t_warm = 0.0;
  for (int k = 0; k < n_batches; ++k) {
    for (int r = 0; r < robots; ++r) order[r] = r;
    // The b oldest requests, in submission order, ties by robot index.
    std::partial_sort(order.begin(), order.begin() + b, order.end(), [&](int x, int y) {
      return submit[x] < submit[y] || (submit[x] == submit[y] && x < y);
    });
    const double start = std::max(free_at, submit[order[b - 1]]);
    const double done = start + batch_ms;
    for (int i = 0; i < b; ++i) {
      const int r = order[i];
      if (k >= warm) lat.push_back(done - submit[r]);
      submit[r] = done + t_act_ms;
    }
    free_at = done;
    if (k == warm - 1) t_warm = done;
  }
  const double span_ms = free_at - t_warm;
  o.throughput_hz = span_ms > 0 ? (double)lat.size() * 1000.0 / span_ms : 0.0;
  o.action_rate_hz = o.throughput_hz / robots;
  double sum = 0.0;
  for (double v : lat) sum += v;
  o.latency_mean_ms = sum / (double)lat.size();
  std::sort(lat.begin(), lat.end());
  o.latency_p50_ms = rank_value(lat, 50, 100);
  o.latency_p99_ms = rank_value(lat, 99, 100);
}

bool sim_args_ok(int32_t robots, int32_t batch, double batch_ms, double t_act_ms, int32_t n_batches) {
  return robots >= 1 && batch >= 1 && std::isfinite(batch_ms) && batch_ms > 0 && std::isfinite(t_act_ms) &&
         t_act_ms >= 0 && n_batches >= 2 && n_batches <= 1000000;
}

}  // namespace

extern "C" rosa_status rosa_s1_simulate(int32_t robots, int32_t batch, double batch_ms, double t_act_ms,
                                        int32_t n_batches, rosa_s1_outcome *out) {
  if (!out || !sim_args_ok(robots, batch, batch_ms, t_act_ms, n_batches)) return ROSA_E_INVALID;
  try {
    simulate(robots, batch, batch_ms, t_act_ms, n_batches, *out);
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}

extern "C" rosa_status rosa_s1_select_batch(const int32_t *batch_sizes, const double *batch_ms, int32_t n_sizes,
                                            int32_t robots, double t_act_ms, double slo_ms, int32_t n_batches,
                                            int32_t *best, rosa_s1_outcome *outcomes) {
  if (!batch_sizes || !batch_ms || !best || n_sizes < 1 || n_sizes > 64 || !std::isfinite(slo_ms)) return ROSA_E_INVALID;
  for (int i = 0; i < n_sizes; ++i) {
    if (!sim_args_ok(robots, batch_sizes[i], batch_ms[i], t_act_ms, n_batches)) return ROSA_E_INVALID;
    for (int j = 0; j < i; ++j)
      if (batch_sizes[j] == batch_sizes[i]) return ROSA_E_INVALID;
  }
  try {
    int32_t pick = -1;
    rosa_s1_outcome chosen{};
    for (int i = 0; i < n_sizes; ++i) {
      rosa_s1_outcome o;
      simulate(robots, batch_sizes[i], batch_ms[i], t_act_ms, n_batches, o);
      if (outcomes) outcomes[i] = o;
      const bool ok = o.feasible && (slo_ms <= 0 || o.latency_p99_ms <= slo_ms);
      if (!ok) continue;
      if (pick < 0 || o.throughput_hz > chosen.throughput_hz ||
          (o.throughput_hz == chosen.throughput_hz && o.batch < chosen.batch)) {
        pick = i;
        chosen = o;
      }
    }
    *best = pick;
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}
