"""Write sampled-row expected outputs of the whole block at full size.

Calls only the CPU oracle (``oracle``) and the seeded input generator
(``synth``); nothing here touches the GPU path.  For each workload the oracle
computes the pre-attention steps for every row (self-attention needs all keys
and values) and the rest of the block for a seeded sample of rows that
includes the first and last row and frame boundaries.  Output:
``block_<workload>.npz`` with ``rows`` (int64 global row indices) and ``y``
(float32 block outputs of those rows).

Usage: python tests/golden/make_block_golden.py [workload ...]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import synth  # noqa: E402
from oracle import dit_block as O  # noqa: E402

N_ROWS = 256


def make(name: str) -> str:
    wl = synth.get_workload(name)
    t0 = time.time()
    w = {k: O.decode(v) for k, v in synth.generate_block_inputs(wl).items()}
    rows = synth.generate_sampled_rows(wl, N_ROWS, sample_id=7)
    y = O.block_forward_rows(O.config_from_workload(wl), O.varlen_from_workload(wl), w["x"], w["t"], w["txt"], w,
                             rows, row_chunk=4096)
    out = os.path.join(HERE, f"block_{name}.npz")
    np.savez_compressed(out, rows=rows.astype(np.int64), y=y.astype(np.float32))
    print(f"{name}: {len(rows)} rows in {time.time() - t0:.0f} s -> {out}", flush=True)
    return out


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["video_480p", "video_720p"]):
        make(n)
