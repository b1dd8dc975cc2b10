"""The library's migration planner (dit_migration_plan) against the planner
oracle on the CPU: identical entries on seeded random layouts of every kind;
the capacity protocol; argument validation."""
import numpy as np
import pytest

from oracle import migrate as M

B = pytest.importorskip("paper_2606_13501_amd.binding")


def _lib():
    import os
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libditblock.so not built")
    return B.lib()


def _as_dicts(entries, n, nd):
    return [{"src_rank": e.src_rank, "dst_rank": e.dst_rank, "src_off": list(e.src_off[:nd]),
             "dst_off": list(e.dst_off[:nd]), "extent": list(e.extent[:nd]), "bytes": e.bytes}
            for e in entries[:n]]


def _random_boxes(rng, shape, n_ranks_base):
    """A partition of the shape into a grid of boxes (random cuts per dimension), ranks shuffled."""
    cuts = []
    for s in shape:
        k = int(rng.integers(1, min(4, s) + 1)) if s > 0 else 1
        c = sorted(set([0, s] + [int(x) for x in rng.integers(0, s + 1, k - 1)])) if s > 0 else [0, 0]
        cuts.append(c)
    boxes = []
    import itertools
    for idx in itertools.product(*[range(len(c) - 1) for c in cuts]):
        boxes.append(([cuts[d][i] for d, i in enumerate(idx)], [cuts[d][i + 1] for d, i in enumerate(idx)]))
    ranks = rng.permutation(len(boxes)) + n_ranks_base
    return [(int(r), a, b) for r, (a, b) in zip(ranks, boxes)]


@pytest.mark.parametrize("seed", range(200))
def test_plan_parity_random(seed):
    _lib()
    rng = np.random.default_rng([13501, 88, seed])
    nd = int(rng.integers(1, 5))
    shape = [int(x) for x in rng.integers(1, 9, nd)]
    eb = int(rng.choice([1, 2, 4, 8, 16]))
    kind = int(rng.choice([0, 0, 0, 1, 2]))
    if kind == M.REPLICATED:
        src = [(int(r), [0] * nd, shape) for r in rng.choice(8, int(rng.integers(1, 4)), replace=False)]
        dst = [(int(r), [0] * nd, shape) for r in rng.choice(8, int(rng.integers(1, 6)), replace=False)]
    else:
        src = _random_boxes(rng, shape, 0)
        dst = _random_boxes(rng, shape, int(rng.integers(0, 3)))
        if rng.uniform() < 0.3:      # destinations needing overlapping or partial regions
            dst = dst[: max(1, len(dst) // 2)] + [(99, [0] * nd, shape)]
    ref = M.plan(kind, shape, eb, src, dst)
    f = B.MigField(kind, shape, eb, src, dst)
    entries, n = B.migration_plan(f)
    assert _as_dicts(entries, n, nd) == ref


def test_sp_row_layout_parity():
    _lib()
    for d1 in (1, 2, 4, 8):
        for d2 in (1, 2, 3, 4, 8):
            src = M.row_layout(75600, list(range(d1)), [64])
            dst = M.row_layout(75600, list(range(8, 8 + d2)), [64])
            f = B.MigField(M.SHARDED, (75600, 64), 2, src, dst)
            entries, n = B.migration_plan(f)
            assert _as_dicts(entries, n, 2) == M.plan(M.SHARDED, (75600, 64), 2, src, dst)


def test_capacity_and_validation():
    L = _lib()
    import ctypes
    src = M.row_layout(10, [0, 1], [2])
    dst = M.row_layout(10, [4, 5, 6, 7], [2])
    f = B.MigField(M.SHARDED, (10, 2), 4, src, dst)
    n = ctypes.c_int64(0)
    assert L.dit_migration_plan(ctypes.byref(f.c), None, 0, ctypes.byref(n)) == B.DIT_ERR_WORKSPACE and n.value == 4
    small = (B.CMigEntry * 2)()
    assert L.dit_migration_plan(ctypes.byref(f.c), small, 2, ctypes.byref(n)) == B.DIT_ERR_WORKSPACE
    for bad, msg in [(dict(shape=(9, 2)), "src slice 1"), (dict(elem_bytes=3), "elem_bytes"),
                     (dict(kind=5), "kind"), (dict(src=[]), "no source")]:
        args = dict(kind=M.SHARDED, shape=(10, 2), elem_bytes=4, src=src, dst=dst)
        args.update(bad)
        with pytest.raises(B.DitError) as e:
            B.migration_plan(B.MigField(args["kind"], args["shape"], args["elem_bytes"], args["src"], args["dst"]))
        assert msg in str(e.value), (bad, str(e.value))
    with pytest.raises(B.DitError):
        B.migration_plan(B.MigField(M.REPLICATED, (3, 5), 4, [(0, [0, 0], [3, 4])], [(1, [0, 0], [3, 5])]))
