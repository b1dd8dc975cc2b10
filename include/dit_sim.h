/*
 * dit_sim.h -- C ABI of the trajectory-task simulator (host code, no GPU).
 *
 * The paper's runtime decomposes a request into trajectory tasks, one per
 * denoising step, and a policy decides which ready task runs next and on how
 * many ranks (section 3.2).  Its simulator keeps the task graph and the policy
 * interface but takes completion events from a cost table of profiled task
 * latencies indexed by task type, request shape and parallel configuration
 * (section 5.5), to compare policies offline.  The three policies are those of
 * section 5.4: FCFS with workload-aware group assignment, SRTF with per-rank
 * (here: per-group) local queues, EDF with best-fit parallelism.
 *
 * The simulated unit is the denoising step: a request is a chain of n_steps
 * steps, each running without preemption on d ranks for cost(class, d).  All
 * times are integer microseconds.  Rules (in this order at each time t):
 *  1. every step ending at t completes, in order of request id: it frees its
 *     ranks, then finishes the request at t or makes its next step ready;
 *  2. every request arriving at t becomes ready, in order of id;
 *  3. the policy dispatches ready steps onto free ranks.
 * Policies:
 *  - DIT_SIM_FCFS_GROUPS: fixed groups of group_size consecutive ranks; a step
 *    that becomes ready joins the group with the least queued work (remaining
 *    time of its running step + queued step costs; ties: lowest group); an idle
 *    group runs its queued step of the earliest-arrived request (ties: id).
 *  - DIT_SIM_SRTF_GROUPS: groups as above; a request is bound at arrival to
 *    the group with the least remaining work of its unfinished requests (ties:
 *    lowest group); an idle group runs the ready step of its request with the
 *    least remaining work (steps not yet started x step cost; ties: arrival,
 *    id).  group_size 1 is the paper's per-rank SRTF.
 *  - DIT_SIM_EDF_BESTFIT: ready steps by deadline (none last; ties: arrival,
 *    id); each, while ranks are free, gets the smallest degree <= free ranks
 *    whose predicted finish now + (steps not started) x cost <= deadline, or,
 *    if none, the degree with the earliest predicted finish (ties: smaller);
 *    it takes the lowest-numbered free ranks.  The degree can change at every
 *    step (latent migration is free here).
 *
 * Every array is HOST memory, read or written during the call only.  The call
 * is synchronous, allocates only host memory that it frees before returning,
 * and keeps no state.  Errors: DIT_ERR_INVALID_ARG for a bad argument (nothing
 * is written), and the message in dit_last_error().
 */
#ifndef DIT_SIM_H
#define DIT_SIM_H

#include <stdint.h>

#include "dit_block.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { DIT_SIM_FCFS_GROUPS = 0, DIT_SIM_SRTF_GROUPS = 1, DIT_SIM_EDF_BESTFIT = 2 } dit_sim_policy;

typedef struct {
  int n_ranks;             /* G >= 1 */
  int n_degrees;           /* 1..16 */
  const int32_t *degrees;  /* host [n_degrees]: strictly increasing, degrees[0] == 1 */
  int n_classes;           /* >= 1 */
  const int64_t *cost_us;  /* host [n_classes][n_degrees]: one step's latency, > 0 */
  dit_sim_policy policy;
  int group_size;          /* FCFS/SRTF: ranks per group, one of degrees, <= n_ranks */
} dit_sim_config;

typedef struct {
  int64_t n_req;               /* >= 0 */
  const int64_t *arrival_us;   /* host [n_req], >= 0 */
  const int32_t *cls;          /* host [n_req], 0..n_classes-1 */
  const int32_t *n_steps;      /* host [n_req], >= 1 */
  const int64_t *deadline_us;  /* host [n_req] or NULL; a negative entry means none */
} dit_sim_trace;

typedef struct {
  int64_t *finish_us;       /* host [n_req]: completion time of the last step */
  int64_t *first_start_us;  /* host [n_req]: start of the first step */
  int64_t *dispatches;      /* host [n_degrees]: steps run at each degree */
  int64_t events;           /* completion and arrival events processed */
} dit_sim_result;

/* Replay `trace` under `cfg` (rules above) and fill `out`.  The total work,
 * sum of n_steps x the largest cost, plus the last arrival must stay below
 * 2^62 us. */
dit_status dit_simulate(const dit_sim_config *cfg, const dit_sim_trace *trace, dit_sim_result *out);

#ifdef __cplusplus
}
#endif

#endif /* DIT_SIM_H */
