"""Helpers of the GPU parity tests: upload seeded inputs, download results,
and the tolerance checks (fp32: max |g - r| <= 1e-4; bf16: cosine >= 0.9999
and ||g - r||_inf / ||r||_inf <= 2e-2)."""
import os
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import dit_block as O

FP32_MAX_ABS = 1e-4
BF16_MIN_COS = 0.9999
BF16_MAX_REL = 2e-2


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13501_amd.binding as B
    B.lib()   # raises when the HIP library is missing: no silent fallback
    return B


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray) -> torch.Tensor:
    """Stored host array (uint16 = bf16 bits, float32) -> device tensor."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float64 numpy."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def empty(shape, dtype):
    return torch.empty(shape, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")


def stats(g, r):
    g = np.asarray(g, np.float64).ravel()
    r = np.asarray(r, np.float64).ravel()
    d = g - r
    ninf = np.abs(r).max() if r.size else 0.0
    cos = float(np.dot(g, r) / (np.linalg.norm(g) * np.linalg.norm(r))) if r.size and np.linalg.norm(r) > 0 else 1.0
    return {"max_abs": float(np.abs(d).max()) if d.size else 0.0,
            "max_rel": float(np.abs(d).max() / ninf) if ninf > 0 else float(np.abs(d).max() if d.size else 0.0),
            "cos": cos}


def check(g, r, dtype, what):
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU output"
    s = stats(g, r)
    log(f"  parity {what}: max_abs={s['max_abs']:.3e} max_rel={s['max_rel']:.3e} cos={s['cos']:.7f}")
    if dtype == "f32":
        assert s["max_abs"] <= FP32_MAX_ABS, f"{what}: max_abs {s['max_abs']:.3e} > {FP32_MAX_ABS}"
    else:
        assert s["cos"] >= BF16_MIN_COS, f"{what}: cos {s['cos']:.7f} < {BF16_MIN_COS}"
        assert s["max_rel"] <= BF16_MAX_REL, f"{what}: max_rel {s['max_rel']:.3e} > {BF16_MAX_REL}"
    return s


class DeviceBlock:
    """A workload's weights and inputs on the device plus the C structs."""

    def __init__(self, wl, inputs=None, names=None):
        B = require_gpu()
        self.B = B
        self.wl = wl
        self.inp = inputs if inputs is not None else synth.generate_block_inputs(wl, names)
        self.d = {k: dev(v) for k, v in self.inp.items()}
        tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.cfg = B.BlockConfig(wl.hidden, wl.n_heads, wl.head_dim, wl.mlp_hidden, wl.freq_dim,
                                 wl.rope_sections, tdt, rope_theta=wl.rope_theta, ln_eps=wl.ln_eps,
                                 rms_eps=wl.rms_eps)
        self.w = B.make_weights(self.d)
        self.vl = B.Varlen(wl.cu_seqlens(), wl.cu_txt(), list(wl.grids))
        self.ws = torch.empty(B.block_workspace_size(self.cfg, self.vl), dtype=torch.uint8, device="cuda")

    def forward(self, x=None, y=None):
        x = self.d["x"] if x is None else x
        y = torch.empty_like(x) if y is None else y
        self.B.block_forward(self.cfg, self.w, self.vl, x, self.d["t"], self.d["txt"], y, self.ws)
        return y

    def oracle_weights(self):
        return {k: O.decode(v) for k, v in self.inp.items()}


# ---------------------------------------------------------------- sampled rows


def oracle_pre_rows(wl, w, mod, rows):
    """Oracle pre-attention outputs (q, k, v) of the given global rows: each
    row is evaluated as its own one-row request at its grid position."""
    cfg = O.config_from_workload(wl)
    cu = wl.cu_seqlens()
    req = np.searchsorted(np.asarray(cu), rows, side="right") - 1
    vl = O.Varlen(list(range(len(rows) + 1)), [0] * (len(rows) + 1), [wl.grids[r] for r in req],
                  [int(rows[i] - cu[req[i]]) for i in range(len(rows))])
    return O.pre_attention(cfg, vl, w["x"][rows], w, mod[req])


def oracle_post_rows(wl, w, mod, o, rows):
    """Oracle post-attention outputs of the given global rows (attention
    output ``o`` indexed by global row), request by request with its text."""
    cfg = O.config_from_workload(wl)
    cu = wl.cu_seqlens()
    cut = wl.cu_txt()
    out = np.empty((len(rows), wl.hidden))
    for r in range(wl.n_req):
        m = np.nonzero((rows >= cu[r]) & (rows < cu[r + 1]))[0]
        if len(m) == 0:
            continue
        vl = O.Varlen([0, len(m)], [0, cut[r + 1] - cut[r]], [wl.grids[r]])
        out[m] = O.post_attention(cfg, vl, w["x"][rows[m]], o[rows[m]], w["txt"][cut[r]:cut[r + 1]], w,
                                  mod[r:r + 1])
    return out
