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

// ------------------------------------------------------------------ homogeneous scheduling

namespace {

struct RatePointSim {
  uint64_t state;
  uint64_t next() {   // SplitMix64
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
};

void rate_point(int b, double batch_ms, double rate_hz, int n_requests, uint64_t seed, double pct,
                double &mean, double &slo) {
  RatePointSim g{seed};
  std::vector<double> arr(n_requests);
  double t = 0.0;
  for (int i = 0; i < n_requests; ++i) {
    const double u = ((double)(g.next() >> 11) + 0.5) / 9007199254740992.0;
    t += -std::log(u) * 1000.0 / rate_hz;
    arr[i] = t;
  }
  const int n_batches = n_requests / b;
  std::vector<double> lat;
  lat.reserve((size_t)n_requests);
  double free_at = 0.0;
  for (int j = 0; j < n_batches; ++j) {
    const double start = std::max(free_at, arr[(size_t)j * b + b - 1]);
    const double done = start + batch_ms;
    free_at = done;
    if (j >= n_batches / 10)
      for (int i = 0; i < b; ++i) lat.push_back(done - arr[(size_t)j * b + i]);
  }
  double sum = 0.0;
  for (double v : lat) sum += v;
  mean = sum / (double)lat.size();
  std::sort(lat.begin(), lat.end());
  const long n = (long)lat.size();
  long r = (long)std::ceil(pct * (double)n);
  r = std::max(1L, std::min(n, r));
  slo = lat[r - 1];
}

// (mean, slo) of one batch size's profile at a load; false if infeasible.
bool lookup(const rosa_config_profile &c, double load, double &mean, double &slo) {
  const rosa_rate_point *p = c.points;
  const int n = c.n_points;
  if (load > p[n - 1].rate_hz) return false;
  if (load <= p[0].rate_hz) {
    if (load < p[0].rate_hz && c.batch != 1) return false;
    mean = p[0].mean_ms;
    slo = p[0].slo_ms;
    return true;
  }
  for (int i = 0; i + 1 < n; ++i) {
    if (p[i].rate_hz <= load && load <= p[i + 1].rate_hz) {
      const double w = (load - p[i].rate_hz) / (p[i + 1].rate_hz - p[i].rate_hz);
      mean = p[i].mean_ms + w * (p[i + 1].mean_ms - p[i].mean_ms);
      slo = p[i].slo_ms + w * (p[i + 1].slo_ms - p[i].slo_ms);
      return true;
    }
  }
  return false;
}

struct Cfg { int batch, k; double mean, slo; };

std::vector<Cfg> feasible_configs(const rosa_model_profile &m, double per_stream_hz, int robots) {
  const int kmax = m.max_streams > 0 ? std::min(robots, m.max_streams) : robots;
  std::vector<Cfg> out;
  for (int c = 0; c < m.n_configs; ++c)
    for (int k = 1; k <= kmax; ++k) {
      double mean, slo;
      if (lookup(m.configs[c], k * per_stream_hz, mean, slo) && slo <= m.deadline_ms)
        out.push_back({m.configs[c].batch, k, mean, slo});
    }
  return out;
}

// Exact covers of `robots` streams by configurations, one per server: for every
// server count n <= max_servers, the least stream-weighted latency sum
// (sum of k * mean) of a cover with exactly n servers (+inf if none), and the
// covers themselves on request.
struct CoverTable {
  int robots = 0, max_servers = 0;
  std::vector<double> best;        // [n][j]
  std::vector<int> choice;         // [n][j]: configuration of the n-th server
  double at(int n, int j) const { return best[(size_t)n * (robots + 1) + j]; }
};

CoverTable cover_table(const std::vector<Cfg> &cfgs, int robots, int max_servers) {
  CoverTable t;
  t.robots = robots;
  t.max_servers = max_servers;
  const size_t W = (size_t)robots + 1;
  t.best.assign((size_t)(max_servers + 1) * W, INFINITY);
  t.choice.assign((size_t)(max_servers + 1) * W, -1);
  t.best[0] = 0.0;
  for (int n = 1; n <= max_servers; ++n)
    for (int j = 1; j <= robots; ++j) {
      double b = INFINITY;
      int ch = -1;
      for (size_t c = 0; c < cfgs.size(); ++c) {
        const int k = cfgs[c].k;
        if (k > j) continue;
        const double prev = t.best[(size_t)(n - 1) * W + (j - k)];
        if (prev == INFINITY) continue;
        const double v = prev + k * cfgs[c].mean;
        if (v < b) { b = v; ch = (int)c; }
      }
      t.best[(size_t)n * W + j] = b;
      t.choice[(size_t)n * W + j] = ch;
    }
  return t;
}

void unwind(const CoverTable &t, const std::vector<Cfg> &cfgs, int n, std::vector<Cfg> &out) {
  int j = t.robots;
  const size_t W = (size_t)t.robots + 1;
  for (; n > 0; --n) {
    const Cfg &c = cfgs[t.choice[(size_t)n * W + j]];
    out.push_back(c);
    j -= c.k;
  }
}

bool profile_ok(const rosa_model_profile &m) {
  if (m.role < ROSA_ROLE_S1 || m.role > ROSA_ROLE_OBLIGATION || m.max_streams < 0 || m.reserved != 0 ||
      !(m.deadline_ms > 0) || !std::isfinite(m.deadline_ms) || m.n_configs < 1 || m.n_configs > 64 || !m.configs)
    return false;
  if (m.role == ROSA_ROLE_OBLIGATION && (!(m.rate_per_robot_hz > 0) || !std::isfinite(m.rate_per_robot_hz)))
    return false;
  for (int c = 0; c < m.n_configs; ++c) {
    const rosa_config_profile &p = m.configs[c];
    if (p.batch < 1 || p.n_points < 1 || p.n_points > 1000 || !p.points) return false;
    for (int d = 0; d < c; ++d)
      if (m.configs[d].batch == p.batch) return false;
    for (int i = 0; i < p.n_points; ++i) {
      const rosa_rate_point &q = p.points[i];
      if (!(q.rate_hz > 0) || !std::isfinite(q.rate_hz) || !std::isfinite(q.mean_ms) || !std::isfinite(q.slo_ms))
        return false;
      if (i > 0 && !(q.rate_hz > p.points[i - 1].rate_hz)) return false;
    }
  }
  return true;
}

}  // namespace

extern "C" rosa_status rosa_rate_profile(int32_t batch, double batch_ms, int32_t n_rates, int32_t n_requests,
                                         uint64_t seed, double pct, rosa_rate_point *out) {
  if (!out || batch < 1 || !(batch_ms > 0) || !std::isfinite(batch_ms) || n_rates < 1 || n_rates > 100 ||
      n_requests > 10000000 || (int64_t)n_requests < 10 * (int64_t)batch || !(pct > 0) || pct > 1)
    return ROSA_E_INVALID;
  try {
    const double peak = batch * 1000.0 / batch_ms;
    for (int j = 1; j <= n_rates; ++j) {
      const double rate = peak * j / n_rates;
      out[j - 1].rate_hz = rate;
      rate_point(batch, batch_ms, rate, n_requests, seed + (uint64_t)j, pct, out[j - 1].mean_ms, out[j - 1].slo_ms);
    }
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}

extern "C" rosa_status rosa_schedule_homogeneous(const rosa_fleet *fleet, const rosa_model_profile *models,
                                                 int32_t n_models, rosa_fleet_schedule *out,
                                                 rosa_server_plan *servers_out) {
  if (!fleet || !models || !out || n_models < 1 || n_models > 16) return ROSA_E_INVALID;
  const rosa_fleet &F = *fleet;
  if (F.robots < 1 || F.robots > 4096 || F.servers < 1 || F.servers > 1024 || !(F.t_act_ms > 0) ||
      !std::isfinite(F.t_act_ms) || F.horizon < 1 || F.reserved != 0 || !(F.eps_hz > 0) || !std::isfinite(F.eps_hz))
    return ROSA_E_INVALID;
  int64_t n_cfg = 0;
  for (int m = 0; m < n_models; ++m) {
    if (!profile_ok(models[m])) return ROSA_E_INVALID;
    n_cfg += models[m].n_configs;
  }
  // Packing work per search step: servers x robots x (configurations x robots).
  if ((int64_t)F.servers * F.robots * F.robots * n_cfg > (int64_t)40000000000) return ROSA_E_UNSUPPORTED;
  try {
    *out = rosa_fleet_schedule{};
    const int R = F.robots;
    // Step 1: obligation footprints.
    std::vector<rosa_server_plan> plan;
    int used = 0;
    for (int m = 0; m < n_models; ++m) {
      if (models[m].role != ROSA_ROLE_OBLIGATION) continue;
      const std::vector<Cfg> cfgs = feasible_configs(models[m], models[m].rate_per_robot_hz, R);
      const int cap = F.servers - used;
      const CoverTable t = cover_table(cfgs, R, cap);
      int n = 1;
      while (n <= cap && t.at(n, R) == INFINITY) ++n;
      if (n > cap) return ROSA_OK;                    // infeasible
      std::vector<Cfg> got;
      unwind(t, cfgs, n, got);
      for (const Cfg &c : got) plan.push_back({m, c.batch, c.k, 0, c.mean, c.slo});
      used += n;
    }
    out->obligation_servers = used;
    const int budget = F.servers - used;
    std::vector<int> goal;
    for (int m = 0; m < n_models; ++m)
      if (models[m].role != ROSA_ROLE_OBLIGATION) goal.push_back(m);
    const int G = (int)goal.size();
    const double H = (double)F.horizon;

    // Step 2: binary search on f.
    double lo = 0.0, hi = 1000.0 / F.t_act_ms;
    bool have = false;
    std::vector<rosa_server_plan> best_goal;
    double best_f = 0, best_l1 = 0, best_l2 = 0, best_loop = 0;
    int steps = 0;
    while (hi - lo > F.eps_hz) {
      const double f = (lo + hi) / 2;
      ++steps;
      // Step 2.1 + 2.2: per goal model the best latency sum for each server
      // count, then the cheapest split of the budget over the models.
      std::vector<std::vector<Cfg>> cfgs(G);
      std::vector<CoverTable> tabs(G);
      for (int g = 0; g < G; ++g) {
        const rosa_model_profile &m = models[goal[g]];
        cfgs[g] = feasible_configs(m, m.role == ROSA_ROLE_S1 ? f : f / H, R);
        tabs[g] = cover_table(cfgs[g], R, budget);
      }
      // acc[g][t]: least cost of models 0..g-1 with t servers in total; pick[g][t]: servers of model g-1.
      std::vector<std::vector<double>> acc(G + 1, std::vector<double>(budget + 1, INFINITY));
      std::vector<std::vector<int>> pick(G + 1, std::vector<int>(budget + 1, -1));
      acc[0][0] = 0.0;
      for (int g = 0; g < G; ++g) {
        const double w = models[goal[g]].role == ROSA_ROLE_S1 ? 1.0 : 1.0 / H;
        for (int t = 0; t <= budget; ++t) {
          if (acc[g][t] == INFINITY) continue;
          for (int n = 1; t + n <= budget; ++n) {
            const double s = tabs[g].at(n, R);
            if (s == INFINITY) continue;
            const double v = acc[g][t] + w * (s / R);
            if (v < acc[g + 1][t + n]) { acc[g + 1][t + n] = v; pick[g + 1][t + n] = n; }
          }
        }
      }
      int tb = -1;
      for (int t = 0; t <= budget; ++t)
        if (acc[G][t] < INFINITY && (tb < 0 || acc[G][t] < acc[G][tb])) tb = t;
      bool ok = false;
      double l1 = 0, l2 = 0, loop = 0;
      std::vector<rosa_server_plan> gplan;
      if (tb >= 0) {
        int t = tb;
        std::vector<int> ns(G);
        for (int g = G; g >= 1; --g) { ns[g - 1] = pick[g][t]; t -= pick[g][t]; }
        for (int g = 0; g < G; ++g) {
          std::vector<Cfg> got;
          unwind(tabs[g], cfgs[g], ns[g], got);
          const double l = tabs[g].at(ns[g], R) / R;
          if (models[goal[g]].role == ROSA_ROLE_S1) l1 += l;
          else l2 += l;
          for (const Cfg &c : got) gplan.push_back({goal[g], c.batch, c.k, 0, c.mean, c.slo});
        }
        loop = 1000.0 / (F.t_act_ms + l1 + l2 / H);
        ok = f <= loop;
      }
      if (ok) {
        have = true;
        best_f = f; best_l1 = l1; best_l2 = l2; best_loop = loop;
        best_goal.swap(gplan);
        lo = f;
      } else {
        hi = f;
      }
    }
    out->steps = steps;
    if (!have) return ROSA_OK;
    out->feasible = 1;
    out->f_hz = best_f;
    out->l_s1_ms = best_l1;
    out->l_s2_ms = best_l2;
    out->f_loop_hz = best_loop;
    out->goal_servers = (int32_t)best_goal.size();
    if (servers_out) {
      size_t i = 0;
      for (const auto &p : plan) servers_out[i++] = p;
      for (const auto &p : best_goal) servers_out[i++] = p;
    }
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}
