"""The simulator oracle against its pins, and planted mistakes in it (on the
CPU) that at least one pin must catch."""
import pytest

from oracle import sim as S
from oracle_sim_pins import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=[c.__name__ for c in ALL_CHECKS])
def test_pin(check):
    check()


def _patched(src_old, src_new):
    """A copy of oracle.sim.simulate with one line of its source changed."""
    import inspect
    import textwrap
    src = inspect.getsource(S.simulate)
    assert src_old in src, src_old
    ns = dict(vars(S))
    exec(textwrap.dedent(src.replace(src_old, src_new, 1)), ns)
    return ns["simulate"]


# (Ties between groups are broken towards the lowest group, but the groups are
# identical, so that choice only relabels groups and no output depends on it.)
MUTANTS = {
    "fcfs_latest_first": ("key=lambda q: (arrival[q], q))", "key=lambda q: (-arrival[q], q))"),
    "srtf_longest_first": ("key=lambda q: ((n_steps[q] - started[q]) * cost(q, g), arrival[q], q))",
                           "key=lambda q: (-(n_steps[q] - started[q]) * cost(q, g), arrival[q], q))"),
    "srtf_counts_done_not_started": ("key=lambda q: ((n_steps[q] - started[q]) * cost(q, g)",
                                     "key=lambda q: ((n_steps[q] - done[q]) * cost(q, g) * 0 + arrival[q] * 0"),
    "edf_ignores_deadline": ("key=lambda q: (dl[q] < 0, max(dl[q], 0), arrival[q], q))",
                             "key=lambda q: (arrival[q], q))"),
    "edf_largest_meeting": ("d = meet[0]", "d = meet[-1]"),
    "edf_no_regrowth": ("d = min(allowed, key=lambda x: (now + rem * cost(i, x), x))", "d = allowed[0]"),
    "edf_remaining_off_by_one": ("rem = n_steps[i] - started[i]", "rem = n_steps[i] - started[i] - 1"),
    "group_cost_at_degree_1": ("running[i] = (now + cost(i, degree), where, degree)",
                               "running[i] = (now + cost(i, 1), where, degree)"),
    "fcfs_ignores_running_step": ("        if r is not None:\n            w += running[r][0] - now",
                                  "        if r is not None:\n            w += 0"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_caught(monkeypatch, name):
    old, new = MUTANTS[name]
    try:
        mutant = _patched(old, new)
    except AssertionError:
        pytest.fail(f"mutant {name}: source line not found")
    monkeypatch.setattr(S, "simulate", mutant)
    failed = []
    for c in ALL_CHECKS:
        try:
            c()
        except Exception:
            failed.append(c.__name__)
    assert failed, f"no pin catches {name}"
