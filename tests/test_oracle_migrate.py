"""The migration-planner oracle against its pins, and planted mistakes in it
(on the CPU) that at least one pin must catch."""
import inspect
import textwrap

import pytest

from oracle import migrate as M
from oracle_migrate_pins import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=[c.__name__ for c in ALL_CHECKS])
def test_pin(check):
    check()


MUTANTS = {
    "closed_interval": ("if any(hi[d] <= lo[d] for d in range(nd)):", "if any(hi[d] < lo[d] for d in range(nd)):"),
    "offset_from_global": ('"src_off": [lo[d] - ss[d] for d in range(nd)],', '"src_off": [lo[d] for d in range(nd)],'),
    "dst_offset_from_src": ('"dst_off": [lo[d] - ds[d] for d in range(nd)],', '"dst_off": [lo[d] - ss[d] for d in range(nd)],'),
    "start_uses_min": ("lo = [max(ss[d], ds[d]) for d in range(nd)]", "lo = [min(ss[d], ds[d]) for d in range(nd)]"),
    "bytes_ignore_elem": ('"bytes": int(np.prod(ext)) * elem_bytes})', '"bytes": int(np.prod(ext))})'),
    "replicated_first_source": ("k = src_ranks.index(drank) if drank in src_ranks else j % len(src)", "k = 0"),
    "source_major_order": ("    for drank, ds, de in dst:\n        for srank, ss, se in src:",
                           "    for srank, ss, se in src:\n        for drank, ds, de in dst:"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_caught(monkeypatch, name):
    old, new = MUTANTS[name]
    src = inspect.getsource(M.plan)
    assert old in src, name
    ns = dict(vars(M))
    exec(textwrap.dedent(src.replace(old, new, 1)), ns)
    monkeypatch.setattr(M, "plan", ns["plan"])
    failed = []
    for c in ALL_CHECKS:
        try:
            c()
        except Exception:
            failed.append(c.__name__)
    assert failed, f"no pin catches {name}"
