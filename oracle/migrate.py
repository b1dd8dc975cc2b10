"""CPU oracle of the layout-aware migration planner -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU baseline leg of
``bench.py`` may import it; the library's planner shares no code with it.

What it computes.  When two adjacent trajectory tasks use different execution
layouts, the runtime rebuilds each artifact under the new layout (section 5.3,
Layout-Aware Artifact Migration).  From the source and destination views of a
field -- replicated, sharded or metadata-only, with a global shape and a
per-rank slice for tensors -- the planner intersects every source-owned slice
with every destination-required slice; each non-empty intersection is a
transfer of (source rank, destination rank, source range, destination range,
byte size).

Readings (M1..M5):
 M1 a slice is a half-open box [start, end) per dimension of the global shape
    (at most 4 dimensions), stored row-major and densely on its rank;
 M2 entries come destination by destination (in the order the destination
    slices are given), and within one destination source by source (in the
    order given); ranges are offsets inside the source and destination slices
    plus a common extent;
 M3 a replicated field: each destination receives the whole tensor from the
    source with the same rank if there is one, else from source (j mod n_src)
    for the j-th destination (spreading the senders);
 M4 a metadata-only field moves no tensor data: no entries;
 M5 entries with a zero extent are not emitted.

Pins (tests/test_oracle_migrate.py): applying the plan rebuilds the
destination exactly as direct slicing of the global tensor does; a
partitioning source layout covers every destination element exactly once and
moves exactly the destination's bytes; identical layouts move each slice to
its own rank in one entry; a hand-worked SP2 -> SP4 plan.
"""
from typing import Dict, List, Sequence, Tuple

import numpy as np

SHARDED, REPLICATED, METADATA = 0, 1, 2


def plan(kind: int, shape: Sequence[int], elem_bytes: int, src: Sequence[Tuple[int, Sequence[int], Sequence[int]]],
         dst: Sequence[Tuple[int, Sequence[int], Sequence[int]]]) -> List[Dict[str, object]]:
    """src, dst: lists of (rank, start, end) boxes.  Returns the transfer entries."""
    nd = len(shape)
    out = []
    if kind == METADATA:
        return out
    if kind == REPLICATED:
        src_ranks = [s[0] for s in src]
        for j, (drank, _, _) in enumerate(dst):
            k = src_ranks.index(drank) if drank in src_ranks else j % len(src)
            out.append({"src_rank": src[k][0], "dst_rank": drank, "src_off": [0] * nd, "dst_off": [0] * nd,
                        "extent": list(shape), "bytes": int(np.prod(shape)) * elem_bytes})
        return out
    for drank, ds, de in dst:
        for srank, ss, se in src:
            lo = [max(ss[d], ds[d]) for d in range(nd)]
            hi = [min(se[d], de[d]) for d in range(nd)]
            if any(hi[d] <= lo[d] for d in range(nd)):
                continue
            ext = [hi[d] - lo[d] for d in range(nd)]
            out.append({"src_rank": srank, "dst_rank": drank,
                        "src_off": [lo[d] - ss[d] for d in range(nd)],
                        "dst_off": [lo[d] - ds[d] for d in range(nd)],
                        "extent": ext, "bytes": int(np.prod(ext)) * elem_bytes})
    return out


def apply(entries, src_arrays: Dict[int, np.ndarray], dst_shapes: Dict[int, Sequence[int]], dtype) -> Dict[int, np.ndarray]:
    """Execute a plan on host arrays: every entry copies its box from the
    source rank's slice array into the destination rank's slice array."""
    out = {r: np.zeros(s, dtype=dtype) for r, s in dst_shapes.items()}
    for e in entries:
        sl_s = tuple(slice(o, o + x) for o, x in zip(e["src_off"], e["extent"]))
        sl_d = tuple(slice(o, o + x) for o, x in zip(e["dst_off"], e["extent"]))
        out[e["dst_rank"]][sl_d] = src_arrays[e["src_rank"]][sl_s]
    return out


def row_layout(n_rows: int, ranks: Sequence[int], width: Sequence[int] = ()) -> List[Tuple[int, List[int], List[int]]]:
    """Sequence-parallel row layout: rank i of d owns rows [ceil(n*i/d), ceil(n*(i+1)/d)) (the
    trailing dimensions whole)."""
    d = len(ranks)
    out = []
    for i, r in enumerate(ranks):
        a, b = -(-n_rows * i // d), -(-n_rows * (i + 1) // d)
        out.append((r, [a] + [0] * len(width), [b] + list(width)))
    return out
