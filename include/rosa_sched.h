/*
 * rosa_sched.h - profiling-guided System-1 batch-size selection and
 * homogeneous fleet scheduling (host only).
 *
 * The paper's scheduler picks a discrete batch size for each System-1
 * (action-model) server from measured latency profiles, because a larger
 * batch raises the server's throughput but adds latency and queueing to every
 * robot's control loop (Sec. 3.4.1 and Sec. 3.4.2, Step 2.1, per-server
 * configurations built from measured serving profiles; Sec. 4.3, System-1
 * batching).  Robots run closed loop: a robot sends its request, waits for
 * the action chunk, executes it for t_act, then sends the next one, so its
 * action rate is bounded by 1 / (t_act + l_S1) (Sec. 3.4.2, Step 2.3,
 * Eq. scheduler-cycle, with no System-2 term here).
 *
 * Server model used for the choice (the paper gives no queueing model; this
 * is the reading the library takes):
 *  - one GPU worker serving `robots` identical robots with batch size b;
 *  - requests queue in submission order (ties by robot index); a batch starts
 *    when the worker is idle and b requests are waiting, takes the b oldest,
 *    and returns all their chunks after batch_ms (the measured latency of one
 *    rosa_generate_actions call on b requests);
 *  - every robot submits its first request at time 0 and its next one t_act
 *    after its chunk returns;
 *  - with fewer than b robots no batch ever forms (infeasible).
 * The simulation is deterministic.  Statistics cover the requests of the last
 * n_batches / 2 batches (the first half is warm-up): throughput = those
 * requests / (end of the last batch - end of batch n_batches / 2), action
 * rate = throughput / robots, latency = return time - submission time, and
 * percentiles take the value of rank ceil(q n) of the sorted latencies.
 *
 * Same conventions as rosa.h: pure C, noexcept, status returns.
 */
#ifndef ROSA_SCHED_H_
#define ROSA_SCHED_H_

#include "rosa.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rosa_s1_outcome {
  int32_t batch;              /* batch size b */
  int32_t feasible;           /* 1 if batches form (robots >= b), else 0 */
  double  throughput_hz;      /* action chunks per second, all robots */
  double  action_rate_hz;     /* per robot */
  double  latency_mean_ms;
  double  latency_p50_ms;
  double  latency_p99_ms;
} rosa_s1_outcome;

/* Closed-loop simulation of one worker (model above).  robots >= 1,
 * batch >= 1, batch_ms > 0, t_act_ms >= 0, 2 <= n_batches <= 1e6, out != NULL;
 * else ROSA_E_INVALID.  An infeasible case returns ROSA_OK with feasible = 0
 * and zero rates and latencies. */
rosa_status rosa_s1_simulate(int32_t robots, int32_t batch, double batch_ms, double t_act_ms,
                             int32_t n_batches, rosa_s1_outcome *out);

/* Batch-size choice from a measured profile: batch_sizes[i] (distinct, >= 1)
 * with measured call latency batch_ms[i] (> 0), i < n_sizes (1..64).  Every
 * size is simulated; among the feasible ones whose p99 latency is at most
 * slo_ms (slo_ms <= 0: no SLO) the one with the highest throughput wins, ties
 * to the smaller batch.  *best = its index, or -1 if none qualifies.
 * outcomes (may be NULL) receives n_sizes entries in input order. */
rosa_status rosa_s1_select_batch(const int32_t *batch_sizes, const double *batch_ms, int32_t n_sizes,
                                 int32_t robots, double t_act_ms, double slo_ms, int32_t n_batches,
                                 int32_t *best, rosa_s1_outcome *outcomes);

/* ------------------------------------------------------------------------
 * Homogeneous task scheduling: every robot of the fleet runs the same task
 * (Sec. 3.4.2, the homogeneous-scheduling algorithm).
 *  1. Obligation models (safety, monitor: a fixed invocation rate per robot)
 *     get the fewest servers that carry the fleet's streams within their
 *     deadline (ties: the least stream-weighted mean latency).
 *  2. The remaining servers serve the goal-coupled models.  The shared action
 *     rate f is binary-searched in (0, 1000 / t_act_ms]; at a candidate f each
 *     robot sends System-1 requests at f and System-2 requests at f / H.
 *  2.1 Feasible per-server configurations: (model, batch size b, k streams),
 *     1 <= k <= min(robots, max_streams), whose latency at the aggregate load
 *     (k f, or k f / H) is within the model's deadline.
 *  2.2 Exact packing (the paper solves an ILP; here a dynamic program over
 *     servers and streams per model, then over models): every goal model's
 *     `robots` streams are covered with at most the remaining servers,
 *     minimising l_S1 + l_S2 / H, then the number of servers.  l_m is the
 *     stream-weighted mean latency of model m's chosen servers.
 *  2.3 f is accepted when a packing exists and f <= 1000 / (t_act_ms + l_S1 +
 *     l_S2 / H) (Eq. scheduler-cycle); the search stops when the interval is
 *     at most eps_hz wide and returns the last accepted f.
 * Latency profiles L_m(b, lambda) are tables of rosa_rate_point sorted by
 * rate (the paper profiles ten rates, 10% to 100% of the batch size's maximum
 * throughput).  A load between two points takes their linear interpolation;
 * above the last point it is infeasible; below the first point it takes the
 * first point for b = 1 and is infeasible for b > 1 (a batch that waits for b
 * requests waits without bound as the load falls).
 * Cost: O(servers x robots x sum over b of k_max) time and O(servers x
 * robots) memory per model and search step; fleets with servers x robots^2 x
 * (batch sizes over all models) above 4e10 return ROSA_E_UNSUPPORTED.
 */

/* Latency of one batch size at one aggregate request rate. */
typedef struct rosa_rate_point {
  double rate_hz;
  double mean_ms;             /* mean latency */
  double slo_ms;              /* latency at the model's SLO percentile */
} rosa_rate_point;

/* System-1 profile of one batch size from its measured call latency: n_rates
 * points at rates j / n_rates of b * 1000 / batch_ms (j = 1 .. n_rates).
 * Point j simulates n_requests Poisson arrivals: gaps -ln(u) / rate, u = (the
 * top 53 bits of successive SplitMix64 outputs from state seed + j, + 0.5) /
 * 2^53; a batch starts when the server is idle and b requests wait, takes the
 * b oldest and returns them after batch_ms; requests of an incomplete last
 * batch are dropped; statistics cover the batches after the first tenth;
 * slo_ms is the value of rank ceil(pct n) of the sorted latencies.
 * batch >= 1, batch_ms > 0, 1 <= n_rates <= 100, n_requests >= 10 batch and
 * <= 1e7, 0 < pct <= 1; else ROSA_E_INVALID. */
rosa_status rosa_rate_profile(int32_t batch, double batch_ms, int32_t n_rates, int32_t n_requests, uint64_t seed,
                              double pct, rosa_rate_point *out);

enum { ROSA_ROLE_S1 = 0, ROSA_ROLE_S2 = 1, ROSA_ROLE_OBLIGATION = 2 };

/* Profile of one batch size of a model: n_points points sorted by rate. */
typedef struct rosa_config_profile {
  int32_t batch;
  int32_t n_points;
  const rosa_rate_point *points;
} rosa_config_profile;

typedef struct rosa_model_profile {
  int32_t role;               /* ROSA_ROLE_* */
  int32_t max_streams;        /* most robot streams one server holds (memory); 0: no bound */
  double  deadline_ms;        /* bound on slo_ms */
  double  rate_per_robot_hz;  /* obligation models: each robot's invocation rate */
  int32_t n_configs;
  int32_t reserved;           /* must be 0 */
  const rosa_config_profile *configs;
} rosa_model_profile;

typedef struct rosa_fleet {
  int32_t robots;             /* 1 <= |R| <= 4096 */
  int32_t servers;            /* 1 <= |S| <= 1024 (GPU workers, one model each) */
  double  t_act_ms;           /* action execution time > 0 */
  int32_t horizon;            /* H >= 1: S1 actions per S2 plan */
  int32_t reserved;           /* must be 0 */
  double  eps_hz;             /* search resolution > 0 */
} rosa_fleet;

/* One server of the schedule. */
typedef struct rosa_server_plan {
  int32_t model;              /* index into models */
  int32_t batch;
  int32_t streams;            /* robots it serves */
  int32_t reserved;
  double  mean_ms;            /* at its load */
  double  slo_ms;
} rosa_server_plan;

typedef struct rosa_fleet_schedule {
  int32_t feasible;           /* 1 if some f was accepted */
  int32_t obligation_servers;
  int32_t goal_servers;
  int32_t steps;              /* binary-search steps taken */
  double  f_hz;               /* the shared action rate */
  double  l_s1_ms, l_s2_ms;   /* stream-weighted mean latencies at f */
  double  f_loop_hz;          /* 1000 / (t_act + l_S1 + l_S2 / H) at f */
} rosa_fleet_schedule;

/* The schedule (algorithm above).  models: n_models (1..16) profiles, at most
 * one per batch size each, with at least one goal model unless all are
 * obligations.  servers_out (may be NULL) receives obligation_servers +
 * goal_servers entries (at most fleet->servers), obligation models first, in
 * model order.  Errors: ROSA_E_INVALID for bad arguments (unsorted or
 * non-finite points, duplicate batch sizes, nonzero reserved fields);
 * ROSA_E_NOMEM.  An infeasible fleet returns ROSA_OK with feasible = 0. */
rosa_status rosa_schedule_homogeneous(const rosa_fleet *fleet, const rosa_model_profile *models, int32_t n_models,
                                      rosa_fleet_schedule *out, rosa_server_plan *servers_out);

#ifdef __cplusplus
}
#endif

#endif /* ROSA_SCHED_H_ */
