/*
 * rosa_sched.h - profiling-guided System-1 batch-size selection (host only).
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

#ifdef __cplusplus
}
#endif

#endif /* ROSA_SCHED_H_ */
