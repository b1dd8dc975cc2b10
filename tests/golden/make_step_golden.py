"""Write sampled-token expected outputs of one denoising step at full size.

Calls only the CPU oracle (``oracle``) and the seeded input generator
(``synth``); nothing here touches the GPU path.  The step is the 480p video
step workload cut to its first block (the per-block work is that of the
40-block step): the oracle patch-embeds every token, runs the block's
pre-attention steps on every row (self-attention needs all keys and values)
and the rest of the block, the output layer and the velocity on a seeded
sample of tokens that includes the first and last token and frame boundaries.
Output: ``<step workload>_1block.npz`` with ``rows`` (int64 token indices) and
``v`` (float32 velocity of those tokens, patch order (c, i, j, k)); the Euler
update of those tokens is latent + dt * v.

Usage: python tests/golden/make_step_golden.py [step workload ...]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import synth  # noqa: E402
from oracle import dit_block as O  # noqa: E402
from oracle import dit_model as M  # noqa: E402

N_ROWS = 32


def make(name: str) -> str:
    mw = synth.get_model_workload(name)
    wl = mw.block
    t0 = time.time()
    model, blocks = synth.generate_model_inputs(mw, n_blocks=1)
    mo = {k: O.decode(v) for k, v in model.items()}
    w = {k: O.decode(v) for k, v in blocks[0].items()}
    cfg, vl = O.config_from_workload(wl), O.varlen_from_workload(wl)
    rows = synth.generate_sampled_rows(wl, N_ROWS, sample_id=9)
    tok = M.patchify_packed(mo["latent"], mw.in_channels, list(wl.grids), mw.patch)
    x = O.linear(tok, mo["w_pe"], mo["b_pe"])
    c = M.shared_time(mo["t"], cfg.freq_dim, mo)
    mod = O.adaln_modulation(c, w["w_ada"], w["b_ada"])
    y = O.block_forward_rows(cfg, vl, x, mo["t"], mo["txt"], w, rows, mod=mod, row_chunk=4096)
    req = np.searchsorted(np.asarray(wl.cu_seqlens()), rows, side="right") - 1
    v = M.final_layer(y, c, req, cfg.ln_eps, mo)
    out = os.path.join(HERE, f"{name}_1block.npz")
    np.savez_compressed(out, rows=rows.astype(np.int64), v=v.astype(np.float32))
    print(f"{name}: {len(rows)} tokens in {time.time() - t0:.0f} s -> {out}", flush=True)
    return out


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["step_video_480p", "step_video_720p"]):
        make(n)
