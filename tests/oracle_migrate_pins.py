"""Pins of the migration-planner oracle (``oracle.migrate``): rebuilding a
destination layout from a plan equals slicing the global tensor directly;
partitioning layouts cover every element once and move exactly the
destination's bytes; identical layouts are rank-local; a plan worked out by
hand; replicated and metadata fields."""
import numpy as np

from oracle import migrate as M


def _slices(global_t, layout):
    return {r: global_t[tuple(slice(a, b) for a, b in zip(s, e))].copy() for r, s, e in layout}


def _rebuild_equals_direct(shape, src, dst, seed):
    g = np.random.default_rng(seed).standard_normal(shape).astype(np.float32)
    plan = M.plan(M.SHARDED, shape, 4, src, dst)
    got = M.apply(plan, _slices(g, src), {r: [b - a for a, b in zip(s, e)] for r, s, e in dst}, np.float32)
    want = _slices(g, dst)
    for r in want:
        assert np.array_equal(got[r], want[r]), r
    return plan


def check_sp_row_layouts_rebuild():
    """Row layouts of every SP degree into every other (the latent between
    steps of different layouts): the rebuilt slices equal direct slicing, and
    the bytes moved equal the tensor's."""
    n, w = 101, 6
    for d1 in (1, 2, 3, 4, 8):
        for d2 in (1, 2, 4, 5, 8):
            src = M.row_layout(n, list(range(d1)), [w])
            dst = M.row_layout(n, list(range(10, 10 + d2)), [w])
            plan = _rebuild_equals_direct((n, w), src, dst, seed=d1 * 10 + d2)
            assert sum(e["bytes"] for e in plan) == n * w * 4, (d1, d2)


def check_boxes_cover_once():
    """A 3-D tensor split into blocks along two dimensions at the source and
    a different split at the destination: every destination element is written
    by exactly one entry."""
    shape = (4, 9, 7)
    src = [(i * 3 + j, [0, a, b], [4, a2, b2]) for i, (a, a2) in enumerate([(0, 4), (4, 9)])
           for j, (b, b2) in enumerate([(0, 2), (2, 5), (5, 7)])]
    dst = [(20 + i, [a, 0, 0], [a2, 9, 7]) for i, (a, a2) in enumerate([(0, 1), (1, 3), (3, 4)])]
    _rebuild_equals_direct(shape, src, dst, seed=7)
    plan = M.plan(M.SHARDED, shape, 2, src, dst)
    count = {r: np.zeros([b - a for a, b in zip(s, e)], dtype=int) for r, s, e in dst}
    for e in plan:
        count[e["dst_rank"]][tuple(slice(o, o + x) for o, x in zip(e["dst_off"], e["extent"]))] += 1
    assert all((c == 1).all() for c in count.values())
    assert sum(e["bytes"] for e in plan) == 4 * 9 * 7 * 2


def check_identity_layout_is_local():
    """The same layout on both sides: one entry per rank, from itself, whole slice."""
    lay = M.row_layout(50, [3, 1, 2], [4])
    plan = M.plan(M.SHARDED, (50, 4), 2, lay, lay)
    assert len(plan) == 3
    for e, (r, s, en) in zip(plan, lay):
        assert e["src_rank"] == r and e["dst_rank"] == r
        assert e["src_off"] == [0, 0] and e["dst_off"] == [0, 0] and e["extent"] == [en[0] - s[0], 4]


def check_hand_worked_sp2_to_sp4():
    """10 rows: SP2 owns rows 0-5 (rank 0) and 5-10 (rank 1); SP4 on ranks 4..7
    needs rows 0-3, 3-5, 5-8, 8-10.  Destination 5 (rows 3-5) comes from
    rank 0's rows 3-5; destination 6 (rows 5-8) from rank 1's rows 0-3."""
    src = M.row_layout(10, [0, 1], [2])
    dst = M.row_layout(10, [4, 5, 6, 7], [2])
    plan = M.plan(M.SHARDED, (10, 2), 4, src, dst)
    got = [(e["src_rank"], e["dst_rank"], e["src_off"][0], e["dst_off"][0], e["extent"][0]) for e in plan]
    assert got == [(0, 4, 0, 0, 3), (0, 5, 3, 0, 2), (1, 6, 0, 0, 3), (1, 7, 3, 0, 2)], got
    assert [e["bytes"] for e in plan] == [24, 16, 24, 16]


def check_entry_order_follows_destinations():
    """Entries come destination by destination in the order the destination
    slices are listed (here the reverse of the row order)."""
    src = M.row_layout(10, [0, 1], [1])
    dst = [(5, [5, 0], [10, 1]), (4, [0, 0], [5, 1])]
    plan = M.plan(M.SHARDED, (10, 1), 4, src, dst)
    assert [(e["src_rank"], e["dst_rank"]) for e in plan] == [(1, 5), (0, 4)], plan


def check_overlap_straddling():
    """A destination slice straddling two sources gets two entries, in source order."""
    src = M.row_layout(9, [0, 1, 2], [1])          # rows 0-3, 3-6, 6-9
    dst = [(9, [2, 0], [7, 1])]                    # rows 2-7
    plan = M.plan(M.SHARDED, (9, 1), 4, src, dst)
    got = [(e["src_rank"], e["src_off"][0], e["dst_off"][0], e["extent"][0]) for e in plan]
    assert got == [(0, 2, 0, 1), (1, 0, 1, 3), (2, 0, 4, 1)], got


def check_replicated_and_metadata():
    """Replicated: each destination gets the whole tensor once, from its own rank
    when that rank holds a copy, else spread over the sources.  Metadata: nothing."""
    shape = (3, 5)
    src = [(0, [0, 0], [3, 5]), (1, [0, 0], [3, 5])]
    dst = [(1, [0, 0], [3, 5]), (2, [0, 0], [3, 5]), (3, [0, 0], [3, 5]), (4, [0, 0], [3, 5])]
    plan = M.plan(M.REPLICATED, shape, 4, src, dst)
    assert [(e["src_rank"], e["dst_rank"]) for e in plan] == [(1, 1), (1, 2), (0, 3), (1, 4)], plan
    assert all(e["bytes"] == 60 and e["extent"] == [3, 5] for e in plan)
    assert M.plan(M.METADATA, shape, 4, src, dst) == []


ALL_CHECKS = [
    check_sp_row_layouts_rebuild, check_boxes_cover_once, check_identity_layout_is_local,
    check_hand_worked_sp2_to_sp4, check_entry_order_follows_destinations, check_overlap_straddling, check_replicated_and_metadata,
]
