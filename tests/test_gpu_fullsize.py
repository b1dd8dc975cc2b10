"""Parity at full size: the 480p and 720p video blocks (32,760 and 75,600
tokens) and the packed sequence-parallel share (four requests, 5 attention
heads over 121,672 rows), in the launch configuration the benchmark times.

The GPU computes every row; the oracle computes a seeded sample of 2048
rows per request (all rows of a shorter request): the first and last row of
every request, its frame boundaries, the first and last row of every
256-row GEMM tile, and random rows.  Self-attention uses seeded q, k, v; the
stages before and after it (S1-S3, S5-S12) are checked on those rows with a
seeded attention output; the whole block is compared with expected rows
written by tests/golden/make_block_golden.py (oracle only).  The
memory-bound stages are compared on every row."""
import os

import numpy as np
import pytest
import torch

import synth
from oracle import dit_block as O
from gpu_util import DeviceBlock, require_gpu, dev, host, empty, check, log, oracle_pre_rows, oracle_post_rows

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.mark.parametrize("name", ["video_720p", "video_480p", "packed_sp8_share"])
def test_self_attention_full_size(name):
    B = require_gpu()
    wl = synth.get_workload(name)
    H = wl.attn_heads or wl.n_heads
    d = wl.head_dim
    W = H * d
    log(f"case full-size self-attention {name}: rows {wl.cu_attn()[-1]} heads {H}")
    att = synth.generate_attention_inputs(wl)
    T = att["q"].shape[0]
    # three planes [3, T, W], as the block's pre-attention steps write them
    qkv = np.stack([att[n].reshape(T, W) for n in ("q", "k", "v")])
    t = dev(qkv)
    o = empty((T, W), "bf16")
    cu = wl.cu_attn()
    B.attention_varlen(t[0], t[1], t[2], o, cu, cu, H, d)
    torch.cuda.synchronize()
    rows = synth.generate_sampled_rows(wl, 2048, sample_id=3, attn=True)
    g = host(o[torch.from_numpy(rows).cuda()])
    del t, o
    ref = O.attention_varlen(O.decode(qkv[0]), O.decode(qkv[1]), O.decode(qkv[2]), cu, cu, H, d, q_rows=rows)
    check(g, ref, "bf16", f"{name} self-attention ({len(rows)} sampled rows)")


@pytest.mark.parametrize("name", ["video_720p", "video_480p", "packed_sp8_share"])
def test_pre_post_attention_full_size(name):
    wl = synth.get_workload(name)
    log(f"case full-size pre/post attention {name}: rows {wl.n_rows}")
    db = DeviceBlock(wl)
    B = db.B
    T, D = wl.n_rows, wl.hidden
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    qkv = empty((3, T, D), "bf16")
    B.block_pre_attention(db.cfg, db.w, db.vl, db.d["x"], db.d["t"], mod, qkv, db.ws)
    o_in = synth.generate_attention_inputs(wl)["o"]
    y = empty((T, D), "bf16")
    B.block_post_attention(db.cfg, db.w, db.vl, db.d["x"], dev(o_in), db.d["txt"], mod, y, db.ws)
    torch.cuda.synchronize()
    rows = synth.generate_sampled_rows(wl, 2048, sample_id=4, tile=256)
    log(f"  {len(rows)} sampled rows (every 256-row tile's first and last row among them)")
    idx = torch.from_numpy(rows).cuda()
    g_qkv = host(qkv[:, idx])
    g_y = host(y[idx])
    g_mod = host(mod)
    del qkv, y
    w = db.oracle_weights()
    ref_mod = O.conditioning(w["t"], wl.freq_dim, w)
    check(g_mod, ref_mod, "bf16", f"{name} modulation")
    q, k, v = oracle_pre_rows(wl, w, ref_mod, rows)
    check(g_qkv[0], q, "bf16", f"{name} q")
    check(g_qkv[1], k, "bf16", f"{name} k")
    check(g_qkv[2], v, "bf16", f"{name} v")
    ref_y = oracle_post_rows(wl, w, ref_mod, O.decode(o_in), rows)
    x = w["x"][rows]
    check(g_y, ref_y, "bf16", f"{name} post-attention y")
    check(g_y - x, ref_y - x, "bf16", f"{name} post-attention y - x")


@pytest.mark.parametrize("name", ["video_480p", "video_720p"])
def test_block_full_size_vs_golden(name):
    path = os.path.join(GOLDEN, f"block_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    wl = synth.get_workload(name)
    log(f"case full-size block {name}: rows {wl.n_rows}")
    gold = np.load(path)
    rows, ref = gold["rows"], gold["y"].astype(np.float64)
    db = DeviceBlock(wl)
    y = db.forward()
    torch.cuda.synchronize()
    g = host(y[torch.from_numpy(rows).cuda()])
    x = O.decode(db.inp["x"][rows])
    check(g, ref, "bf16", f"{name} block y ({len(rows)} sampled rows)")
    check(g - x, ref - x, "bf16", f"{name} block y - x")


def test_memory_bound_stages_all_rows():
    """The 720p block's memory-bound stages on all 75,600 rows, each on its
    own inputs: modulated LayerNorm (S1, S10) with the GPU's own modulation,
    affine LayerNorm (S6), per-head RMSNorm + 3D rotary on seeded q and k (S3),
    and the standalone gated residual."""
    wl = synth.get_workload("video_720p")
    log(f"case all-row memory-bound stages {wl.name}: rows {wl.n_rows}")
    db = DeviceBlock(wl, names=["x", "t", "txt", "w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada", "g_q", "g_k",
                                "g_ca", "b_ca", "b_o"])
    B = db.B
    T, D, H, d = wl.n_rows, wl.hidden, wl.n_heads, wl.head_dim
    cu = wl.cu_seqlens()
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    B.timestep_modulation(db.cfg, db.w, db.d["t"], mod, db.ws)
    out = empty((T, D), "bf16")
    B.adaln_modulate(db.d["x"], mod[:, 0], mod[:, 1], 6 * D, cu, wl.ln_eps, out)
    torch.cuda.synchronize()
    x = O.decode(db.inp["x"])
    m = host(mod)
    ref = O.modulate(O.layer_norm(x, wl.ln_eps), m[0, 0], m[0, 1])
    check(host(out), ref, "bf16", "modulated LayerNorm, all rows")
    del ref
    B.layer_norm_affine(db.d["x"], db.d["g_ca"], db.d["b_ca"], wl.ln_eps, out)
    torch.cuda.synchronize()
    ref = O.layer_norm(x, wl.ln_eps) * O.decode(db.inp["g_ca"]) + O.decode(db.inp["b_ca"])
    check(host(out), ref, "bf16", "affine LayerNorm, all rows")
    del ref
    z_bits = synth.draw((T, D), (31, 1))
    gate = mod[:, 2]
    B.gated_residual(db.d["x"], dev(z_bits), db.d["b_o"], gate, 6 * D, cu, out)
    torch.cuda.synchronize()
    ref = x + m[0, 2] * (O.decode(z_bits) + O.decode(db.inp["b_o"]))
    check(host(out), ref, "bf16", "gated residual, all rows")
    del ref, out, z_bits
    qk_bits = synth.draw((T, 2 * D), (31, 2))
    qk = dev(qk_bits)
    vl = B.Varlen(cu, wl.cu_txt(), list(wl.grids))
    B.qk_norm_rope(qk[:, :D], qk[:, D:], H, d, db.d["g_q"], db.d["g_k"], wl.rms_eps, wl.rope_sections,
                   wl.rope_theta, vl)
    torch.cuda.synchronize()
    g = host(qk)
    del qk
    cfg, ovl = O.config_from_workload(wl), O.varlen_from_workload(wl)
    u = O.decode(qk_bits)
    for part, gain in ((slice(0, D), "g_q"), (slice(D, 2 * D), "g_k")):
        ref = O.rope_for_rows(O.rms_norm_heads(u[:, part], O.decode(db.inp[gain]), H, d, wl.rms_eps), cfg, ovl)
        check(g[:, part], ref, "bf16", f"RMSNorm + rotary ({gain[-1]}), all rows")
        del ref
