"""Whole-block parity of the HIP path against the CPU oracle (C ABI), plus
the block's invariants run on the GPU."""
import numpy as np
import pytest
import torch

import synth
from synth.workloads import Workload
from oracle import dit_block as O
from gpu_util import DeviceBlock, require_gpu, dev, host, empty, check, log

pytestmark = pytest.mark.gpu

# A small packed bf16 batch: three requests with ragged lengths, different
# grids and text lengths, 3D rotary.  Its Linear weights have std
# 0.02 * sqrt(5120 / 512) so that activations and adaLN gates have the
# magnitudes of the D = 5120 video block (gates ~0.7).  With plain 0.02 at
# D = 512 the gates are ~0.03, y - x is ~50x smaller than y, and rounding the
# exact result once to bf16 already costs cos(y - x) = 0.9994.
SMALL_PACKED = Workload(
    name="small_packed_bf16", wid=50, dtype="bf16", hidden=512, n_heads=4, head_dim=128, mlp_hidden=1024,
    freq_dim=512, rope_sections=(44, 42, 42), grids=((2, 10, 16), (1, 7, 11), (3, 9, 19)), rows=(300, 77, 513),
    txt_len=64, linear_std=0.02 * (5120 / 512) ** 0.5, description="small packed bf16 batch for parity")


# The video blocks' own shape and weight scale (D = 5120, 40 x 128 heads, MLP
# 13824, rotary sections 44/42/42, Linear weights N(0, 0.02^2) as in the
# 480p and 720p configurations) on two short requests (300 and 180 tokens,
# 512 text tokens each), so every row of a config-scale block is compared.
VIDEO_SMALL = Workload(
    name="video_small_d5120", wid=51, dtype="bf16", hidden=5120, n_heads=40, head_dim=128, mlp_hidden=13824,
    freq_dim=5120, rope_sections=(44, 42, 42), grids=((1, 15, 20), (3, 6, 10)), rows=(300, 180), txt_len=512,
    description="two short video requests at the video blocks' width and weight scale")


def _oracle_block(db: DeviceBlock, x=None):
    wl = db.wl
    w = db.oracle_weights()
    cfg = O.config_from_workload(wl)
    vl = O.varlen_from_workload(wl)
    xx = w["x"] if x is None else x
    return O.block_forward(cfg, vl, xx, w["t"], w["txt"], w)


@pytest.mark.parametrize("name", ["tiny_image_fp32", "image_1024", "small_packed_bf16", "video_small_d5120"])
def test_block_parity(name):
    wl = {"small_packed_bf16": SMALL_PACKED, "video_small_d5120": VIDEO_SMALL}.get(name) or synth.get_workload(name)
    log(f"case block parity {name}")
    db = DeviceBlock(wl)
    y = db.forward()
    torch.cuda.synchronize()
    g = host(y)
    ref = _oracle_block(db)
    x = O.decode(db.inp["x"])
    check(g, ref, wl.dtype, f"{name} y")
    check(g - x, ref - x, wl.dtype, f"{name} y - x")


def test_block_seams_compose_to_forward():
    """pre_attention -> attention -> post_attention == block_forward, bitwise."""
    wl = SMALL_PACKED
    log("case seams compose")
    db = DeviceBlock(wl)
    B = db.B
    y_ref = db.forward()
    T, D = wl.n_rows, wl.hidden
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    qkv = empty((3, T, D), "bf16")
    B.block_pre_attention(db.cfg, db.w, db.vl, db.d["x"], db.d["t"], mod, qkv, db.ws)
    o = empty((T, D), "bf16")
    cu = wl.cu_seqlens()
    B.attention_varlen(qkv[0], qkv[1], qkv[2], o, cu, cu, wl.n_heads, wl.head_dim)
    y = empty((T, D), "bf16")
    B.block_post_attention(db.cfg, db.w, db.vl, db.d["x"], o, db.d["txt"], mod, y, db.ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref)


@pytest.mark.parametrize("name", ["small_packed_bf16", "image_1024"])
def test_block_forward_graph_capture(name):
    """dit_block_forward forks the text key/value projection onto the
    library's side stream at its start and joins it before the
    cross-attention, launches no memset and never synchronises, so the call
    can be captured in a HIP graph: three replays (with eager calls in
    between) each equal the eager result bit for bit.  Neither batch splits
    its attention (three requests; the image takes the 4-wave shape), so
    eager and captured calls run the same kernels."""
    wl = {"small_packed_bf16": SMALL_PACKED}.get(name) or synth.get_workload(name)
    log(f"case block forward graph capture {name}")
    db = DeviceBlock(wl)
    y_ref = db.forward()
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    y = torch.empty_like(y_ref)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        db.B.block_forward(db.cfg, db.w, db.vl, db.d["x"], db.d["t"], db.d["txt"], y, db.ws, stream=stream)
    for rep in range(3):
        y.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), f"replay {rep} differs"
        db.forward()
        torch.cuda.synchronize()


def test_block_output_may_alias_input():
    wl = SMALL_PACKED
    log("case y aliases x")
    db = DeviceBlock(wl)
    y_ref = db.forward()
    x = db.d["x"].clone()
    db.forward(x=x, y=x)
    torch.cuda.synchronize()
    assert torch.equal(x, y_ref)


@pytest.mark.parametrize("name", ["tiny_image_fp32", "small_packed_bf16"])
def test_block_zero_gates_identity(name):
    """gate_sa = gate_ff = 0 and W_co = b_co = 0 give y == x bitwise."""
    wl = SMALL_PACKED if name == "small_packed_bf16" else synth.get_workload(name)
    log(f"case zero-gate identity {name}")
    inp = synth.generate_block_inputs(wl)
    D = wl.hidden
    for c in (2, 5):
        inp["w_ada"][c * D:(c + 1) * D] = 0
        inp["b_ada"][c * D:(c + 1) * D] = 0
    inp["w_co"][:] = 0
    inp["b_co"][:] = 0
    db = DeviceBlock(wl, inputs=inp)
    y = db.forward()
    torch.cuda.synchronize()
    assert torch.equal(y, db.d["x"])


def test_block_permutation_equivariance_without_rope():
    base = SMALL_PACKED
    wl = Workload(**{**base.__dict__, "name": "small_packed_norope", "rope_sections": (0, 0, 0)})
    log("case permutation equivariance")
    db = DeviceBlock(wl)
    y = host(db.forward())
    rng = np.random.default_rng(7)
    cu = wl.cu_seqlens()
    perm = np.concatenate([cu[r] + rng.permutation(cu[r + 1] - cu[r]) for r in range(wl.n_req)])
    xp = db.d["x"][torch.from_numpy(perm).cuda()].contiguous()
    yp = host(db.forward(x=xp))
    torch.cuda.synchronize()
    check(yp, y[perm], "bf16", "permuted")


def test_shard_rows_equal_full_rows():
    """A sequence-parallel shard (pos_offset) gives the same pre-attention
    rows as the full request (per-token steps), bitwise."""
    wl = Workload(**{**SMALL_PACKED.__dict__, "name": "one_req", "grids": ((3, 9, 19),), "rows": (513,),
                     "txt_len": 64})
    log("case shard rows")
    db = DeviceBlock(wl)
    B = db.B
    D = wl.hidden
    mod = torch.empty((1, 6, D), dtype=torch.float32, device="cuda")
    full = empty((3, 513, D), "bf16")
    B.block_pre_attention(db.cfg, db.w, db.vl, db.d["x"], db.d["t"], mod, full, db.ws)
    a, b = 171, 342
    vls = B.Varlen([0, b - a], [0, 64], [(3, 9, 19)], [a])
    shard = empty((3, b - a, D), "bf16")
    xs = db.d["x"][a:b].contiguous()
    ws = torch.empty(B.block_workspace_size(db.cfg, vls), dtype=torch.uint8, device="cuda")
    B.block_pre_attention(db.cfg, db.w, vls, xs, db.d["t"], mod, shard, ws)
    torch.cuda.synchronize()
    assert torch.equal(shard, full[:, a:b])


def test_block_forward_with_precomputed_modulation():
    """dit_block_forward with mod given (t NULL, the block's timestep MLP and
    adaLN weights absent) equals the call that computes mod from t, bit for bit."""
    wl = synth.get_workload("image_1024")
    db = DeviceBlock(wl)
    B = db.B
    y_ref = db.forward()
    D = wl.hidden
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    B.timestep_modulation(db.cfg, db.w, db.d["t"], mod, db.ws)
    d2 = dict(db.d)
    for n in ("w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada"):
        d2[n] = None
    y = torch.empty_like(y_ref)
    B.block_forward(db.cfg, B.make_weights(d2), db.vl, db.d["x"], None, db.d["txt"], y, db.ws, mod=mod)
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref)


def test_block_seams_with_precomputed_modulation():
    """The seams take a precomputed modulation like dit_block_forward does:
    pre(mod) -> attention -> post(mod), with the block's timestep MLP and
    adaLN weights absent, equals forward(mod) bit for bit; post(t) (the
    modulation computed inside) equals post(mod) bit for bit."""
    wl = SMALL_PACKED
    log("case seams with precomputed modulation")
    db = DeviceBlock(wl)
    B = db.B
    T, D = wl.n_rows, wl.hidden
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    B.timestep_modulation(db.cfg, db.w, db.d["t"], mod, db.ws)
    d2 = dict(db.d)
    for n in ("w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada"):
        d2[n] = None
    w2 = B.make_weights(d2)
    y_ref = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
    B.block_forward(db.cfg, w2, db.vl, db.d["x"], None, db.d["txt"], y_ref, db.ws, mod=mod)
    mod_in = mod.clone()
    qkv = empty((3, T, D), "bf16")
    B.block_pre_attention(db.cfg, w2, db.vl, db.d["x"], None, mod_in, qkv, db.ws)
    o = empty((T, D), "bf16")
    cu = wl.cu_seqlens()
    B.attention_varlen(qkv[0], qkv[1], qkv[2], o, cu, cu, wl.n_heads, wl.head_dim)
    y = empty((T, D), "bf16")
    B.block_post_attention(db.cfg, w2, db.vl, db.d["x"], o, db.d["txt"], mod_in, y, db.ws)
    y_t = empty((T, D), "bf16")
    B.block_post_attention(db.cfg, db.w, db.vl, db.d["x"], o, db.d["txt"], None, y_t, db.ws, t=db.d["t"])
    torch.cuda.synchronize()
    assert torch.equal(mod_in, mod), "pre_attention with t NULL wrote mod"
    assert torch.equal(y, y_ref)
    assert torch.equal(y_t, y_ref)
