"""Pins of the simulator oracle (``oracle.sim``): a schedule worked out by
hand, closed forms of single-rank schedules, the optimality of SRTF (mean
completion time) and EDF (maximum lateness) on one rank against brute force
over all orders, and the best-fit degree in closed form.  Each ``check_*``
raises AssertionError on a mismatch."""
import itertools

import numpy as np

from oracle import sim as S


def check_fcfs_hand_schedule():
    """Two single-rank groups, costs 100 us at degree 1.  A (2 steps) and B
    (1 step) arrive at 0, C (1 step) at 50.  t=0: A -> group 0, B -> group 1
    (group 0 holds A's 100 us).  t=50: C -> group 0 (both groups 50 us, tie to
    the lowest).  t=100: A's step ends, its second step goes to group 1 (B's
    step ends at 100: 0 us left), B finishes; group 0 starts C, group 1 A.
    t=200: both finish."""
    r = S.simulate(2, [1, 2], [[100, 60]], S.FCFS_GROUPS, 1, [0, 0, 50], [0, 0, 0], [2, 1, 1])
    assert r["finish"] == [200, 100, 200], r
    assert r["first_start"] == [0, 0, 100], r
    assert r["dispatches"] == [4, 0], r
    assert r["events"] == 7, r


def check_fcfs_least_queued_work():
    """The queued work of a group includes what is left of its running step:
    A (1000 us) takes group 0 at 0, B (100 us) group 1 at 10; C (100 us) at 20
    sees 980 us on group 0 and 90 us on group 1, so it waits behind B and
    finishes at 210 (not behind A at 1100)."""
    r = S.simulate(2, [1], [[1000], [100]], S.FCFS_GROUPS, 1, [0, 10, 20], [0, 1, 1], [1, 1, 1])
    assert r["finish"] == [1000, 110, 210], r


def check_fcfs_single_rank_prefix_sums():
    """One rank, everyone at t = 0: FCFS runs the requests to completion in id
    order, so finish times are prefix sums of steps * cost."""
    rng = np.random.default_rng(1)
    costs = [[int(c)] for c in rng.integers(10, 1000, 4)]
    cls = [int(c) for c in rng.integers(0, 4, 9)]
    steps = [int(s) for s in rng.integers(1, 6, 9)]
    r = S.simulate(1, [1], costs, S.FCFS_GROUPS, 1, [0] * 9, cls, steps)
    ref = np.cumsum([steps[i] * costs[cls[i]][0] for i in range(9)]).tolist()
    assert r["finish"] == ref, (r["finish"], ref)


def check_fcfs_single_rank_arrivals():
    """One rank, arrivals spread out: finish_i = max(finish_{i-1}, a_i) + work_i
    in arrival order (the rank never idles while work waits)."""
    rng = np.random.default_rng(2)
    n = 12
    arr = sorted(int(a) for a in rng.integers(0, 5000, n))
    steps = [int(s) for s in rng.integers(1, 5, n)]
    costs = [[300], [170]]
    cls = [i % 2 for i in range(n)]
    r = S.simulate(1, [1], costs, S.FCFS_GROUPS, 1, arr, cls, steps)
    t, ref = 0, []
    for i in range(n):
        t = max(t, arr[i]) + steps[i] * costs[cls[i]][0]
        ref.append(t)
    assert r["finish"] == ref, (r["finish"], ref)


def check_srtf_optimal_mean_completion():
    """One rank, all at t = 0: SRTF minimises the mean completion time; compare
    with the best of all run-to-completion orders."""
    rng = np.random.default_rng(3)
    for trial in range(5):
        n = 6
        costs = [[int(c)] for c in rng.integers(10, 400, n)]
        steps = [int(s) for s in rng.integers(1, 7, n)]
        cls = list(range(n))
        r = S.simulate(1, [1], costs, S.SRTF_GROUPS, 1, [0] * n, cls, steps)
        work = [steps[i] * costs[i][0] for i in range(n)]
        best = min(sum(np.cumsum([work[i] for i in p])) for p in itertools.permutations(range(n)))
        assert sum(r["finish"]) == best, (trial, sum(r["finish"]), best)


def check_edf_optimal_max_lateness():
    """One rank, degree 1 only, all at t = 0: EDF minimises the maximum
    lateness (Jackson's rule); compare with brute force over all orders."""
    rng = np.random.default_rng(4)
    for trial in range(5):
        n = 6
        costs = [[int(c)] for c in rng.integers(10, 300, n)]
        steps = [int(s) for s in rng.integers(1, 5, n)]
        work = [steps[i] * costs[i][0] for i in range(n)]
        dl = [int(d) for d in rng.integers(0, sum(work), n)]
        r = S.simulate(1, [1], costs, S.EDF_BESTFIT, 1, [0] * n, list(range(n)), steps, dl)
        lat = max(r["finish"][i] - dl[i] for i in range(n))
        best = min(max(f - dl[i] for i, f in zip(p, np.cumsum([work[i] for i in p])))
                   for p in itertools.permutations(range(n)))
        assert lat == best, (trial, lat, best)


def check_edf_best_fit_degree():
    """One request alone on 8 ranks, costs 1000/600/350/200 us at degree
    1/2/4/8, 10 steps: the smallest degree whose predicted finish meets the
    deadline; none -> the fastest; no deadline -> degree 1."""
    costs = [[1000, 600, 350, 200]]
    deg = [1, 2, 4, 8]
    for dl, want_deg, want_fin in [(3500, 4, 3500), (2000, 8, 2000), (1000, 8, 2000),
                                   (6000, 2, 6000), (10000, 1, 10000), (-1, 1, 10000)]:
        r = S.simulate(8, deg, costs, S.EDF_BESTFIT, 1, [0], [0], [10], [dl])
        assert r["finish"] == [want_fin], (dl, r)
        assert r["dispatches"][deg.index(want_deg)] == 10, (dl, r)
    # deadline 3499: degree 4 predicts 3500, so the first step takes 8 ranks
    # (ends at 200); then degree 4 predicts 200 + 9 x 350 = 3350 <= 3499, so
    # the remaining 9 steps drop back to 4 ranks
    r = S.simulate(8, deg, costs, S.EDF_BESTFIT, 1, [0], [0], [10], [3499])
    assert r["finish"] == [3350] and r["dispatches"] == [0, 0, 9, 1], r


def check_edf_grows_at_risk():
    """Two requests on 2 ranks: the earlier deadline takes both ranks (degree 2
    is the smallest meeting it), the other waits, then finds itself at risk and
    takes the fastest degree left."""
    costs = [[100, 60]]
    r = S.simulate(2, [1, 2], costs, S.EDF_BESTFIT, 1, [0, 0], [0, 0], [3, 3], [200, 500])
    # request 0: degree 1 predicts 300 > 200, degree 2 predicts 180 -> 2 ranks, 3 x 60 = 180
    # request 1 waits until 180; then degree 1 predicts 480 <= 500 -> 1 rank, done at 480
    assert r["finish"] == [180, 480], r
    assert r["dispatches"] == [3, 3], r


def check_srtf_group_binding():
    """Two single-rank groups: requests bind at arrival to the group with the
    least remaining work and stay there.  A (5 x 100) -> group 0, B (1 x 100)
    -> group 1, C (2 x 100, at 50) -> group 1 (50 us left there against 450).
    Group 1 then runs C after B: B 100, C 300; A 500."""
    r = S.simulate(2, [1], [[100]], S.SRTF_GROUPS, 1, [0, 0, 50], [0, 0, 0], [5, 1, 2])
    assert r["finish"] == [500, 100, 300], r
    assert r["first_start"] == [0, 0, 100], r


def check_srtf_preempts_at_step_boundary():
    """One rank: a long request is overtaken at its next step boundary by a
    shorter one that arrived meanwhile (SRTF acts at trajectory boundaries)."""
    r = S.simulate(1, [1], [[100]], S.SRTF_GROUPS, 1, [0, 150], [0, 0], [5, 1])
    # A runs 0-100, 100-200; B arrives 150 (100 us of work < A's 300 left): B runs 200-300; A ends 600
    assert r["finish"] == [600, 300], r


def check_group_degree_cost():
    """FCFS with groups of 4 ranks runs every step at degree 4's cost."""
    r = S.simulate(8, [1, 2, 4, 8], [[1000, 600, 350, 200]], S.FCFS_GROUPS, 4, [0, 0, 0], [0, 0, 0], [2, 2, 2])
    # two groups: requests 0 and 1 run in parallel (700 each), request 2 waits for the first free group
    assert r["finish"] == [700, 700, 1400], r
    assert r["dispatches"] == [0, 0, 6, 0], r


ALL_CHECKS = [
    check_fcfs_hand_schedule, check_fcfs_least_queued_work, check_fcfs_single_rank_prefix_sums, check_fcfs_single_rank_arrivals,
    check_srtf_optimal_mean_completion, check_edf_optimal_max_lateness, check_edf_best_fit_degree,
    check_edf_grows_at_risk, check_srtf_group_binding, check_srtf_preempts_at_step_boundary,
    check_group_degree_cost,
]
