"""The library's simulator (dit_simulate, native C++) against the simulator
oracle, on the CPU: identical finish times, first starts, per-degree dispatch
counts and event counts on seeded random traces for every policy, the
oracle's pins replayed on the library, and argument validation."""
import numpy as np
import pytest

from oracle import sim as S
import oracle_sim_pins as P

B = pytest.importorskip("paper_2606_13501_amd.binding")


def _lib():
    import os
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libditblock.so not built")
    return B.lib()


def _lib_simulate(n_ranks, degrees, cost_us, policy, group_size, arrival, cls, n_steps, deadline=None):
    r = B.simulate(n_ranks, degrees, cost_us, policy, group_size, arrival, cls, n_steps, deadline)
    return {"finish": r["finish"].tolist(), "first_start": r["first_start"].tolist(),
            "dispatches": r["dispatches"].tolist(), "events": r["events"]}


@pytest.mark.parametrize("check", P.ALL_CHECKS, ids=[c.__name__ for c in P.ALL_CHECKS])
def test_library_passes_oracle_pins(monkeypatch, check):
    _lib()
    monkeypatch.setattr(S, "simulate", _lib_simulate)
    check()


def _random_case(seed):
    rng = np.random.default_rng([13501, 77, seed])
    degrees = [1, 2, 4, 8][: int(rng.integers(1, 5))]
    G = int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
    n_cls = int(rng.integers(1, 5))
    base = rng.integers(50, 3000, n_cls)
    # costs fall with the degree, but not always monotonically (small requests do not scale)
    cost = [[int(max(1, b / d ** rng.uniform(0.0, 1.0) + rng.integers(0, 40))) for d in degrees] for b in base]
    n = int(rng.integers(1, 60))
    arrival = np.sort(rng.integers(0, int(rng.choice([1, 500, 20000])), n)).tolist()   # many ties when small
    perm = rng.permutation(n)          # ids not in arrival order
    arrival = [arrival[i] for i in perm]
    cls = rng.integers(0, n_cls, n).tolist()
    steps = rng.integers(1, 8, n).tolist()
    dl = None
    if rng.uniform() < 0.8:
        dl = [int(a + rng.integers(-100, 20000)) if rng.uniform() < 0.85 else -1 for a in arrival]
    policy = int(rng.integers(0, 3))
    gs = [d for d in degrees if d <= G]
    group = int(rng.choice(gs))
    return G, degrees, cost, policy, group, arrival, cls, steps, dl


@pytest.mark.parametrize("seed", range(300))
def test_parity_random_traces(seed):
    _lib()
    case = _random_case(seed)
    ref = S.simulate(*case)
    got = _lib_simulate(*case)
    assert got == ref, (case, got, ref)


def test_parity_large_trace():
    """A longer trace with the measured-table shape: 6 classes, 4 degrees, 8 ranks."""
    _lib()
    rng = np.random.default_rng(5)
    degrees = [1, 2, 4, 8]
    cost = [[int(c * 1000 / d ** 0.9) for d in degrees] for c in (790, 1467, 5779, 61, 106, 237)]
    n = 400
    arrival = np.sort(rng.integers(0, 40_000_000, n)).tolist()
    cls = rng.integers(0, 6, n).tolist()
    steps = [50] * n
    dl = [a + int(3.0 * 50 * cost[c][0]) for a, c in zip(arrival, cls)]
    for policy, group in [(S.FCFS_GROUPS, 1), (S.FCFS_GROUPS, 4), (S.SRTF_GROUPS, 1), (S.SRTF_GROUPS, 8),
                          (S.EDF_BESTFIT, 1)]:
        args = (8, degrees, cost, policy, group, arrival, cls, steps, dl)
        assert _lib_simulate(*args) == S.simulate(*args), (policy, group)


def test_rejects_bad_arguments():
    _lib()
    ok = dict(n_ranks=2, degrees=[1, 2], cost_us=[[100, 60]], policy=0, group_size=1, arrival_us=[0],
              cls=[0], n_steps=[1])
    B.simulate(**ok)
    for bad, msg in [(dict(degrees=[2, 4]), "degrees[0]"), (dict(degrees=[1, 1], cost_us=[[1, 1]]), "increase"),
                     (dict(cost_us=[[100, 0]]), "cost_us"), (dict(group_size=3), "group_size"),
                     (dict(group_size=2, n_ranks=1), "n_ranks"), (dict(cls=[1]), "cls"),
                     (dict(n_steps=[0]), "n_steps"), (dict(arrival_us=[-5]), "arrival"),
                     (dict(policy=7), "policy"), (dict(n_ranks=0), "n_ranks")]:
        args = dict(ok, **bad)
        with pytest.raises(B.DitError) as e:
            B.simulate(**args)
        assert e.value.status == B.DIT_ERR_INVALID_ARG and msg in str(e.value), (bad, str(e.value))


def test_empty_trace():
    _lib()
    r = B.simulate(4, [1, 2], [[10, 6]], 2, 1, [], [], [])
    assert r["events"] == 0 and r["dispatches"].tolist() == [0, 0]
