"""The no-workspace conditioning entry point (dit_timestep_modulation_noalloc)
against the workspace one (dit_timestep_modulation), through the C ABI: the
same kernels, so the results must be equal bit for bit.  Two calls in a row
on the shared static scratch, the second with fewer requests, each checked;
also against the oracle, to the bf16 bar."""
import numpy as np
import pytest
import torch

import synth
from oracle import dit_block as O
from gpu_util import DeviceBlock, check, host, log

pytestmark = pytest.mark.gpu

COND = ["t", "w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada"]


@pytest.mark.parametrize("name", ["video_720p", "image_1024"])
def test_noalloc_modulation_matches_workspace_entry(name):
    wl = synth.get_workload(name)
    log(f"case no-alloc modulation {name}")
    db = DeviceBlock(wl, names=COND + ["x", "txt"])
    B = db.B
    D = wl.hidden
    w = db.oracle_weights()
    for n_req in (7, 3):   # the second call is smaller and reuses the scratch
        t = synth.draw((n_req,), (77, n_req), dtype="f32", dist="uniform", lo=0.0, hi=1000.0)
        td = torch.from_numpy(t).cuda()
        ref = torch.full((n_req, 6, D), float("nan"), dtype=torch.float32, device="cuda")
        got = torch.full((n_req, 6, D), float("nan"), dtype=torch.float32, device="cuda")
        B.timestep_modulation(db.cfg, db.w, td, ref, db.ws)
        B.timestep_modulation_noalloc(db.cfg, db.w, td, got)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"{name}: no-alloc modulation differs ({n_req} requests)"
        check(host(got), O.conditioning(t.astype(np.float64), wl.freq_dim, w), "bf16",
              f"{name} no-alloc modulation, {n_req} requests")
