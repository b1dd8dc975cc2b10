"""CPU oracle of the trajectory-task simulator -- TEST INFRASTRUCTURE ONLY.

Like the other oracle modules, only the tests, ``__graft_entry__.smoke()``
and the CPU baseline leg of ``bench.py`` may import it; the library's
simulator shares no code with it.

What it computes.  The paper runs a request as a chain of trajectory tasks and
lets a policy choose, whenever tasks are ready and ranks are free, which task
runs next and on how many ranks (section 3.2); its simulator replaces the
workers with completion events taken from a cost table of profiled task
latencies indexed by task type, request shape and parallel configuration
(section 5.5).  The three policies are the ones it evaluates (section 5.4):
FCFS with workload-aware group assignment, SRTF with per-rank local queues,
EDF with best-fit parallelism.  The paper gives their intent, not their
arithmetic; the readings below fix it.  Every quantity is an integer number
of microseconds, so the oracle and the library agree exactly.

Readings (S1..S9):
 S1 tasks: a request is a chain of n_steps denoising steps; step s + 1 is
    ready when step s completes; the encoder and decoder tasks are not
    simulated (their costs are not measured here).  A step runs on a group of
    d ranks for cost[class][d] without preemption.
 S2 events: at a time t, first every step that ends at t completes, in order
    of request id: it frees its ranks, then finishes its request at t or makes
    the request's next step ready (which S3 assigns at that moment); then every
    request arriving at t becomes ready, in order of id; then the policy
    dispatches.
 S3 FCFS-groups(g): the ranks form G div g fixed groups of g consecutive
    ranks.  A step that becomes ready (in the order of S2) is assigned to the
    group with the least queued work -- the remaining time of its running step
    plus the costs of the steps queued on it -- ties to the lowest group.  An
    idle group starts its queued step of the earliest-arrived request (ties by
    id).
 S4 SRTF-groups(g): groups as in S3.  A request is bound at arrival to the
    group with the least queued work -- over the group's unfinished requests,
    the remaining time of a running step plus the cost of every step not yet
    started -- ties to the lowest group; all its steps run there.  An idle
    group starts the ready step of its request with the least remaining
    trajectory work (steps not yet started times the step cost), ties by
    arrival, then id.
 S5 EDF-bestfit: one queue of ready steps in order of deadline (none = last),
    then arrival, then id.  Going down the queue while ranks are free, the step
    gets the smallest allowed degree d <= free ranks whose predicted finish,
    now + (steps not yet started) * cost[class][d], is at most the deadline;
    if none meets it, the allowed degree with the earliest predicted finish
    (ties to the smaller).  It takes the lowest-numbered free ranks.  The
    degree may change from step to step (migration of the latent between
    layouts costs nothing here).
 S6 costs come from the measured cost table: step latency per (class, degree);
    degree 1 is always allowed.
 S7 outputs: per request its finish time and the start of its first step; per
    degree the number of steps run at it; the number of completion and arrival
    events processed.
 S8 deadlines: the trace gives each request a scheduler-visible deadline
    (a + alpha_c * T_c in the paper, T_c its standalone service time); a
    negative deadline means none.
 S9 a group or rank set is idle exactly when its last step has completed.

Pins (tests/test_oracle_sim.py): hand-computed schedules, single-rank FCFS
prefix sums, SRTF against brute force over all orders (mean completion time),
EDF against brute force over all orders (maximum lateness), work
conservation, best-fit degree choice in closed form.
"""
from typing import Dict, List, Optional, Sequence

FCFS_GROUPS, SRTF_GROUPS, EDF_BESTFIT = 0, 1, 2
NO_DEADLINE = None


def simulate(n_ranks: int, degrees: Sequence[int], cost_us: Sequence[Sequence[int]], policy: int,
             group_size: int, arrival: Sequence[int], cls: Sequence[int], n_steps: Sequence[int],
             deadline: Optional[Sequence[int]] = None) -> Dict[str, object]:
    """Replay a trace under one policy.  cost_us[c][k] is the step latency of
    class c at degrees[k].  Returns finish, first_start (lists per request),
    dispatches (per degree) and events."""
    n = len(arrival)
    dl = [(-1 if deadline is None else deadline[i]) for i in range(n)]
    kof = {d: k for k, d in enumerate(degrees)}

    def cost(i, d):
        return cost_us[cls[i]][kof[d]]

    done = [0] * n                 # steps completed
    started = [0] * n              # steps started
    finish = [-1] * n
    first = [-1] * n
    ready = [False] * n
    dispatches = [0] * len(degrees)
    events = 0
    # running steps: request -> (end time, group index or rank list, degree)
    running: Dict[int, tuple] = {}

    g = group_size
    n_groups = n_ranks // g if policy in (FCFS_GROUPS, SRTF_GROUPS) else 0
    group_busy = [None] * n_groups          # request running on the group, or None
    group_queue: List[List[int]] = [[] for _ in range(n_groups)]   # FCFS: requests whose ready step is queued
    bound = [-1] * n                        # SRTF: group of the request
    free_ranks = set(range(n_ranks))        # EDF

    def queued_work_fcfs(j, now):
        w = 0
        r = group_busy[j]
        if r is not None:
            w += running[r][0] - now
        for q in group_queue[j]:
            w += cost(q, g)
        return w

    def queued_work_srtf(j, now):
        w = 0
        for i in range(n):
            if bound[i] == j and finish[i] < 0:
                if i in running:
                    w += running[i][0] - now
                w += (n_steps[i] - started[i]) * cost(i, g)
        return w

    def make_ready(i, now):
        ready[i] = True
        if policy == FCFS_GROUPS:
            loads = [queued_work_fcfs(j, now) for j in range(n_groups)]
            j = loads.index(min(loads))
            group_queue[j].append(i)

    def start(i, now, degree, where):
        if first[i] < 0:
            first[i] = now
        ready[i] = False
        started[i] += 1
        dispatches[kof[degree]] += 1
        running[i] = (now + cost(i, degree), where, degree)

    def dispatch(now):
        if policy == FCFS_GROUPS:
            for j in range(n_groups):
                if group_busy[j] is None and group_queue[j]:
                    i = min(group_queue[j], key=lambda q: (arrival[q], q))
                    group_queue[j].remove(i)
                    group_busy[j] = i
                    start(i, now, g, j)
        elif policy == SRTF_GROUPS:
            for j in range(n_groups):
                if group_busy[j] is None:
                    cands = [i for i in range(n) if bound[i] == j and ready[i]]
                    if cands:
                        i = min(cands, key=lambda q: ((n_steps[q] - started[q]) * cost(q, g), arrival[q], q))
                        group_busy[j] = i
                        start(i, now, g, j)
        else:
            order = sorted([i for i in range(n) if ready[i]],
                           key=lambda q: (dl[q] < 0, max(dl[q], 0), arrival[q], q))
            for i in order:
                f = len(free_ranks)
                if f == 0:
                    break
                allowed = [d for d in degrees if d <= f]
                rem = n_steps[i] - started[i]
                meet = [d for d in allowed if dl[i] < 0 or now + rem * cost(i, d) <= dl[i]]
                if meet:
                    d = meet[0]
                else:
                    d = min(allowed, key=lambda x: (now + rem * cost(i, x), x))
                ranks = sorted(free_ranks)[:d]
                for r in ranks:
                    free_ranks.remove(r)
                start(i, now, d, ranks)

    arrived = [False] * n
    while True:
        times = [arrival[i] for i in range(n) if not arrived[i]] + [v[0] for v in running.values()]
        if not times:
            break
        now = min(times)
        for i in sorted(r for r, v in running.items() if v[0] == now):
            _, where, degree = running.pop(i)
            events += 1
            done[i] += 1
            if policy in (FCFS_GROUPS, SRTF_GROUPS):
                group_busy[where] = None
            else:
                free_ranks.update(where)
            if done[i] == n_steps[i]:
                finish[i] = now
            else:
                make_ready(i, now)
        for i in range(n):
            if not arrived[i] and arrival[i] == now:
                arrived[i] = True
                events += 1
                if policy == SRTF_GROUPS:
                    loads = [queued_work_srtf(j, now) for j in range(n_groups)]
                    bound[i] = loads.index(min(loads))
                make_ready(i, now)
        dispatch(now)
    return {"finish": finish, "first_start": first, "dispatches": dispatches, "events": events}
