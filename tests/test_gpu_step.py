"""One denoising step on the GPU (dit_denoise_step, dit_text_kv, dit_patchify,
dit_unpatchify_euler) against the step oracle, plus its invariants at the
720p video size.  Tolerances: fp32 max |g - r| <= 1e-4; bf16 cosine >= 0.9999
and max relative error <= 2e-2, on the next latent and on its update
latent_out - latent (where all of the model's signal is)."""
import os

import numpy as np
import pytest
import torch

import synth
from gpu_util import check, dev, host, log, require_gpu
from oracle import dit_block as O
from oracle import dit_model as M

pytestmark = pytest.mark.gpu


class DeviceStep:
    """A step workload's weights and inputs on the device plus the C structs."""

    def __init__(self, mw, n_blocks=None, inputs=None):
        B = require_gpu()
        self.B, self.mw = B, mw
        wl = mw.block
        self.n_blocks = n_blocks or mw.n_blocks
        self.model, self.blocks = inputs if inputs is not None else synth.generate_model_inputs(mw, n_blocks=n_blocks)
        self.blocks = self.blocks[:self.n_blocks]
        self.dm = {k: dev(v) for k, v in self.model.items()}
        self.db = [{k: dev(v) for k, v in b.items()} for b in self.blocks]
        tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        bc = B.BlockConfig(wl.hidden, wl.n_heads, wl.head_dim, wl.mlp_hidden, wl.freq_dim, wl.rope_sections, tdt,
                           rope_theta=wl.rope_theta, ln_eps=wl.ln_eps, rms_eps=wl.rms_eps)
        self.cfg = B.ModelConfig(bc, self.n_blocks, mw.in_channels, mw.patch)
        self.w = B.ModelWeights(self.dm, [B.make_weights(b) for b in self.db])
        self.vl = B.Varlen(wl.cu_seqlens(), wl.cu_txt(), list(wl.grids))
        self.ws = torch.empty(B.denoise_workspace_size(self.cfg, self.vl), dtype=torch.uint8, device="cuda")
        self.kv = torch.empty(B.text_kv_elems(self.cfg, self.vl), dtype=tdt, device="cuda")
        B.text_kv(self.cfg, self.w, self.vl, self.dm["txt"], self.kv)

    def step(self, latent=None, dt=None, out=None):
        latent = self.dm["latent"] if latent is None else latent
        dt = self.dm["dt"] if dt is None else dt
        out = torch.empty_like(latent) if out is None else out
        self.B.denoise_step(self.cfg, self.w, self.vl, latent, self.dm["t"], dt, self.kv, out, self.ws)
        return out

    def oracle(self, latent=None, dt=None):
        wl = self.mw.block
        cfg = O.config_from_workload(wl)
        vl = O.varlen_from_workload(wl)
        mw = {k: O.decode(v) for k, v in self.model.items()}
        blocks = [{k: O.decode(v) for k, v in b.items()} for b in self.blocks]
        lat = mw["latent"] if latent is None else latent
        dts = mw["dt"] if dt is None else dt
        return M.denoise_step(cfg, vl, self.mw.in_channels, self.mw.patch, lat, mw["t"], dts, mw["txt"], mw, blocks)


STEP_CASES = ["step_tiny_fp32", "step_small_bf16"]


@pytest.mark.parametrize("name", STEP_CASES)
def test_step_vs_oracle(name):
    mw = synth.get_model_workload(name)
    log(f"[step] {name}: {mw.n_blocks} blocks, rows {mw.block.rows}, P {mw.patch_len}")
    s = DeviceStep(mw)
    g = host(s.step())
    torch.cuda.synchronize()
    r = s.oracle()
    lat = O.decode(s.model["latent"])
    check(g, r, mw.block.dtype, f"{name} latent_out")
    check(g - lat, r - lat, mw.block.dtype, f"{name} update")


@pytest.mark.parametrize("name", STEP_CASES)
def test_text_kv_vs_oracle(name):
    mw = synth.get_model_workload(name)
    s = DeviceStep(mw)
    kv = host(s.kv).reshape(s.n_blocks, mw.block.n_txt, 2 * mw.block.hidden)
    cfg = O.config_from_workload(mw.block)
    ref = M.text_kv(cfg, O.decode(s.model["txt"]), [{k: O.decode(v) for k, v in b.items()} for b in s.blocks])
    for b in range(s.n_blocks):
        check(kv[b], ref[b], mw.block.dtype, f"{name} text kv block {b}")


@pytest.mark.parametrize("name", STEP_CASES)
def test_patchify_exact(name):
    """Patchify moves values: bit-exact (bf16 rounds to nearest even)."""
    mw = synth.get_model_workload(name)
    B = require_gpu()
    s = DeviceStep(mw, n_blocks=1)
    tok = torch.empty((mw.block.n_rows, mw.patch_len), dtype=s.kv.dtype, device="cuda")
    B.patchify(s.cfg, s.vl, s.dm["latent"], tok)
    ref = M.patchify_packed(O.decode(s.model["latent"]), mw.in_channels, list(mw.block.grids), mw.patch)
    ref32 = ref.astype(np.float32)
    if mw.block.dtype == "bf16":
        got = tok.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, synth.bf16_bits(ref32)), "bf16 patchify bits"
    else:
        assert np.array_equal(tok.cpu().numpy(), ref32), "fp32 patchify"


@pytest.mark.parametrize("name", STEP_CASES)
@pytest.mark.parametrize("in_place", [False, True])
def test_unpatchify_euler(name, in_place):
    mw = synth.get_model_workload(name)
    B = require_gpu()
    s = DeviceStep(mw, n_blocks=1)
    v_bits = synth.draw((mw.block.n_rows, mw.patch_len), (7, 1), dtype=mw.block.dtype)
    v = dev(v_bits)
    lat = s.dm["latent"].clone()
    out = lat if in_place else torch.empty_like(lat)
    B.unpatchify_euler(s.cfg, s.vl, lat, v, s.dm["dt"], out)
    g = host(out)
    grids = list(mw.block.grids)
    dts = O.decode(s.model["dt"])
    dt_el = np.concatenate([np.full(n, d) for n, d in zip(mw.latent_sizes(), dts)])
    r = M.euler_step(O.decode(s.model["latent"]), M.unpatchify_packed(O.decode(v_bits), mw.in_channels, grids,
                                                                     mw.patch), dt_el)
    err = np.abs(g - r).max()
    log(f"  {name} unpatchify+Euler in_place={in_place}: max abs {err:.2e}")
    assert err <= 4e-6, err      # one fp32 rounding of values below 8


def test_step_packed_equals_alone():
    """Requests never interact: each request stepped alone gives the same bits."""
    mw = synth.get_model_workload("step_small_bf16")
    B = require_gpu()
    s = DeviceStep(mw)
    full = s.step().cpu().numpy()
    wl = mw.block
    cu, cut, sizes = wl.cu_seqlens(), wl.cu_txt(), mw.latent_sizes()
    off = 0
    for r in range(wl.n_req):
        vl = B.Varlen([0, wl.rows[r]], [0, wl.txt_len], [wl.grids[r]])
        ws = torch.empty(B.denoise_workspace_size(s.cfg, vl), dtype=torch.uint8, device="cuda")
        kv = torch.empty(B.text_kv_elems(s.cfg, vl), dtype=s.kv.dtype, device="cuda")
        # clone(): fresh, aligned allocations (a slice keeps its parent's offset)
        B.text_kv(s.cfg, s.w, vl, s.dm["txt"][cut[r]:cut[r + 1]].clone(), kv)
        lat = s.dm["latent"][off:off + sizes[r]].clone()
        out = torch.empty_like(lat)
        B.denoise_step(s.cfg, s.w, vl, lat, s.dm["t"][r:r + 1].clone(), s.dm["dt"][r:r + 1].clone(), kv, out, ws)
        assert np.array_equal(out.cpu().numpy(), full[off:off + sizes[r]]), f"request {r} alone differs"
        off += sizes[r]


def test_step_in_place_and_cache_reuse():
    """latent_out may alias latent; the text cache is read-only, so a second
    step with the same cache and inputs gives the same bits."""
    mw = synth.get_model_workload("step_tiny_fp32")
    s = DeviceStep(mw)
    kv0 = s.kv.clone()
    a = s.step()
    b = s.step()
    lat = s.dm["latent"].clone()
    s.step(latent=lat, out=lat)
    assert torch.equal(a, b), "two steps differ"
    assert torch.equal(lat, a), "in-place step differs"
    assert torch.equal(kv0, s.kv), "the step wrote to the text cache"


@pytest.mark.parametrize("name", ["step_video_720p"])
def test_step_fullsize_properties(name):
    """At the 720p size with 2 of the 40 blocks (the per-block work is the
    bench's): dt = 0 returns the latent bit for bit, the update is linear in
    dt up to one fp32 rounding, outputs are finite, and patchify at this size
    is bit-exact against the oracle."""
    mw = synth.get_model_workload(name)
    B = require_gpu()
    log(f"[step] {name}: generating inputs")
    s = DeviceStep(mw, n_blocks=2)
    lat = s.dm["latent"]
    zero = torch.zeros_like(s.dm["dt"])
    out0 = s.step(dt=zero)
    assert torch.equal(out0, lat), "dt = 0 must return the latent"
    o1 = s.step()
    o2 = s.step(dt=2 * s.dm["dt"])
    d1, d2 = (o1 - lat).double(), (o2 - lat).double()
    assert torch.isfinite(d1).all()
    rel = ((d2 - 2 * d1).abs().max() / d1.abs().max()).item()
    log(f"  {name}: |update| max {d1.abs().max().item():.3e}, linearity residual {rel:.2e}")
    assert rel <= 2e-5, rel
    tok = torch.empty((mw.block.n_rows, mw.patch_len), dtype=torch.bfloat16, device="cuda")
    B.patchify(s.cfg, s.vl, lat, tok)
    ref = M.patchify_packed(O.decode(s.model["latent"]), mw.in_channels, list(mw.block.grids), mw.patch)
    got = tok.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, synth.bf16_bits(ref.astype(np.float32))), "720p patchify bits"


def test_step_graph_capture():
    """The step launches no memset, allocates nothing and never synchronises,
    so it can be captured in a HIP graph: three replays (with eager steps in
    between) each equal the eager result bit for bit."""
    mw = synth.get_model_workload("step_small_bf16")
    s = DeviceStep(mw)
    ref = s.step()
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    out = torch.empty_like(ref)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        s.B.denoise_step(s.cfg, s.w, s.vl, s.dm["latent"], s.dm["t"], s.dm["dt"], s.kv, out, s.ws, stream=stream)
    for rep in range(3):
        out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {rep} differs"
        s.step()
        torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["step_video_480p", "step_video_720p"])
def test_step_fullsize_vs_golden(name):
    """A whole-size step cut to its first block (the per-block work of the
    40-block step): the update latent_out - latent of a seeded sample of
    tokens against the oracle's velocity times dt, from
    tests/golden/make_step_golden.py (oracle only)."""
    mw = synth.get_model_workload(name)
    gold = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"{name}_1block.npz"))
    rows, v = gold["rows"], gold["v"].astype(np.float64)
    log(f"[step] {name} with 1 block vs golden: {len(rows)} tokens")
    s = DeviceStep(mw, n_blocks=1)
    out = s.step().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    grids, C, patch = list(mw.block.grids), mw.in_channels, mw.patch
    lat = O.decode(s.model["latent"])
    upd = (M.patchify_packed(out, C, grids, patch) - M.patchify_packed(lat, C, grids, patch))[rows]
    cu = np.asarray(mw.block.cu_seqlens())
    dts = O.decode(s.model["dt"])[np.searchsorted(cu, rows, side="right") - 1]
    check(upd, dts[:, None] * v, "bf16", f"{name} 1-block update on sampled tokens")
