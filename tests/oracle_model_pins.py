"""Pins of the denoising-step oracle (``oracle.dit_model``): checks against
facts it does not compute itself -- a brute-force patch loop, einops and a
torch Conv3d patch embedding, the flow-matching path, closed forms of special
cases and invariants.  Each ``check_*`` raises AssertionError on a mismatch;
``test_oracle_model.py`` runs them on the oracle as written and on planted
mistakes.  Oracle calls go through the module objects so a patched function
is seen by the step's internal calls too."""
import numpy as np
import torch
import torch.nn.functional as F
from einops import rearrange

from oracle import dit_block as O
from oracle import dit_model as M
from oracle_pins import _close, _t, tiny_setup


def _model_setup(seed=11, C=2, patch=(1, 2, 2), grids=((2, 2, 2), (1, 2, 3)), n_blocks=2, L=3):
    """Tiny packed step: two whole requests, D = 8, two blocks."""
    rows = tuple(g[0] * g[1] * g[2] for g in grids)
    cfg, vl, _, t, txt, _ = tiny_setup(seed=seed, R=len(grids), rows=rows, L=L, grids=grids)
    blocks = [tiny_setup(seed=seed + 1 + b, R=len(grids), rows=rows, L=L, grids=grids)[5]
              for b in range(n_blocks)]
    rng = np.random.default_rng(seed + 100)
    D, P = cfg.hidden, C * patch[0] * patch[1] * patch[2]
    s = 0.3
    mw = {
        "w_t1": rng.standard_normal((D, cfg.freq_dim)) * s, "b_t1": rng.standard_normal(D) * s,
        "w_t2": rng.standard_normal((D, D)) * s, "b_t2": rng.standard_normal(D) * s,
        "w_pe": rng.standard_normal((D, P)) * s, "b_pe": rng.standard_normal(D) * s,
        "w_hmod": rng.standard_normal((2 * D, D)) * s, "b_hmod": rng.standard_normal(2 * D) * s,
        "w_out": rng.standard_normal((P, D)) * s, "b_out": rng.standard_normal(P) * s,
    }
    n_lat = sum(M.latent_sizes(C, grids, patch))
    latent = rng.standard_normal(n_lat)
    dt = -rng.uniform(0.01, 0.1, len(grids))
    return cfg, vl, C, patch, latent, t, dt, txt, mw, blocks


def _step(setup, **kw):
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = setup
    return M.denoise_step(cfg, vl, C, patch, latent, t, dt, txt, mw, blocks, **kw)


# ------------------------------------------------------------ latent <-> tokens


def check_patchify_bruteforce():
    """Every latent value lands at token (f, h, w) row-major, column (c, i, j, k)."""
    rng = np.random.default_rng(1)
    C, (pt, ph, pw), (Fg, Hg, Wg) = 3, (2, 2, 3), (2, 3, 2)
    lat = rng.standard_normal((C, Fg * pt, Hg * ph, Wg * pw))
    tok = M.patchify(lat, (pt, ph, pw))
    ref = np.full((Fg * Hg * Wg, C * pt * ph * pw), np.nan)
    for f in range(Fg):
        for h in range(Hg):
            for w in range(Wg):
                for c in range(C):
                    for i in range(pt):
                        for j in range(ph):
                            for k in range(pw):
                                ref[(f * Hg + h) * Wg + w, ((c * pt + i) * ph + j) * pw + k] = \
                                    lat[c, f * pt + i, h * ph + j, w * pw + k]
    assert np.array_equal(tok, ref), "patchify differs from the brute-force loop"


def check_patchify_einops():
    """The same layout written as an einops pattern (an independent library)."""
    rng = np.random.default_rng(2)
    lat = rng.standard_normal((4, 3 * 1, 2 * 2, 5 * 2))
    ref = rearrange(lat, "c (f i) (h j) (w k) -> (f h w) (c i j k)", i=1, j=2, k=2)
    assert np.array_equal(M.patchify(lat, (1, 2, 2)), ref), "patchify differs from einops"
    tok = rng.standard_normal((3 * 2 * 5, 16))
    ref = rearrange(tok, "(f h w) (c i j k) -> c (f i) (h j) (w k)", f=3, h=2, w=5, c=4, i=1, j=2, k=2)
    assert np.array_equal(M.unpatchify(tok, 4, (3, 2, 5), (1, 2, 2)), ref), "unpatchify differs from einops"


def check_patch_embedding_conv3d():
    """patchify then Linear with W_pe [D, P] equals the standard patch embedding,
    a Conv3d with kernel = stride = patch and weight W_pe viewed as [D, C, pt, ph, pw]."""
    rng = np.random.default_rng(3)
    C, patch, D = 3, (2, 2, 2), 5
    lat = rng.standard_normal((C, 4, 6, 4))
    w = rng.standard_normal((D, C * 8))
    b = rng.standard_normal(D)
    x = O.linear(M.patchify(lat, patch), w, b)
    conv = F.conv3d(_t(lat)[None], _t(w).reshape(D, C, *patch), _t(b), stride=patch)[0]   # [D, F, H, W]
    ref = conv.permute(1, 2, 3, 0).reshape(-1, D).numpy()
    _close(x, ref, 1e-12, "patch embedding vs conv3d")


def check_patch_roundtrip():
    """unpatchify inverts patchify exactly, alone and packed."""
    rng = np.random.default_rng(4)
    grids, patch, C = [(2, 3, 2), (1, 2, 4)], (2, 1, 3), 2
    flat = rng.standard_normal(sum(M.latent_sizes(C, grids, patch)))
    tok = M.patchify_packed(flat, C, grids, patch)
    assert tok.shape == (2 * 3 * 2 + 1 * 2 * 4, C * 6)
    assert np.array_equal(M.unpatchify_packed(tok, C, grids, patch), flat), "packed roundtrip"
    t2 = rng.standard_normal(tok.shape)
    assert np.array_equal(M.patchify_packed(M.unpatchify_packed(t2, C, grids, patch), C, grids, patch), t2)


# ------------------------------------------------------------------ sampler


def check_euler_on_flow_path():
    """On x_s = (1 - s) x0 + s n the exact velocity is n - x0, and one Euler
    step from s to s' lands on x_s' (the path is a straight line)."""
    rng = np.random.default_rng(5)
    x0, n = rng.standard_normal(50), rng.standard_normal(50)
    for s, s2 in [(1.0, 0.96), (0.7, 0.65), (0.1, 0.0)]:
        xs = (1 - s) * x0 + s * n
        _close(M.euler_step(xs, n - x0, s2 - s), (1 - s2) * x0 + s2 * n, 1e-14, f"Euler {s}->{s2}")


def check_final_layer_torch():
    """The final layer against torch: F.silu, F.linear, F.layer_norm."""
    rng = np.random.default_rng(6)
    D, P, R = 8, 6, 2
    x = rng.standard_normal((5, D)) * 2 + 0.5
    c = rng.standard_normal((R, D))
    req = np.array([0, 0, 1, 1, 1])
    mw = {"w_hmod": rng.standard_normal((2 * D, D)), "b_hmod": rng.standard_normal(2 * D),
          "w_out": rng.standard_normal((P, D)), "b_out": rng.standard_normal(P)}
    v = M.final_layer(x, c, req, 1e-6, mw)
    m = F.linear(F.silu(_t(c)), _t(mw["w_hmod"]), _t(mw["b_hmod"]))
    shift, scale = m[:, :D][req], m[:, D:][req]
    h = F.layer_norm(_t(x), (D,), eps=1e-6) * (1 + scale) + shift
    _close(v, F.linear(h, _t(mw["w_out"]), _t(mw["b_out"])).numpy(), 1e-12, "final layer")


# ----------------------------------------------------------------- the step


def check_step_dt_zero():
    """dt = 0 returns the latent unchanged, bit for bit."""
    st = list(_model_setup())
    st[6] = np.zeros_like(st[6])
    assert np.array_equal(_step(st), st[4]), "dt = 0 must leave the latent unchanged"


def check_step_zero_output_weights():
    """W_out = 0: the velocity is b_out in every token, so every latent value
    of channel c at patch offset (i, j, k) moves by dt[r] * b_out[(c,i,j,k)]."""
    st = _model_setup(seed=21)
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = st
    mw["w_out"][:] = 0
    out = _step(st)
    pt, ph, pw = patch
    ref = latent.copy()
    off = 0
    for r, (Fg, Hg, Wg) in enumerate(vl.grid_fhw):
        shape = (C, Fg * pt, Hg * ph, Wg * pw)
        for idx in np.ndindex(*shape):
            c, z, y, x = idx
            col = ((c * pt + z % pt) * ph + y % ph) * pw + x % pw
            ref[off + np.ravel_multi_index(idx, shape)] += dt[r] * mw["b_out"][col]
        off += int(np.prod(shape))
    _close(out, ref, 1e-14, "zero output weights")


def check_step_identity_blocks():
    """Blocks with zero gates and a zero cross output projection are the
    identity, so the step is embedding -> final layer -> Euler, evaluated here
    with torch (layer_norm, silu, linear) and einops."""
    st = _model_setup(seed=31)
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = st
    D = cfg.hidden
    for w in blocks:
        for g in (2, 5):
            w["w_ada"][g * D:(g + 1) * D] = 0
            w["b_ada"][g * D:(g + 1) * D] = 0
        w["w_co"][:] = 0
        w["b_co"][:] = 0
    out = _step(st)
    pt, ph, pw = patch
    e = _t(O.timestep_embedding(t, cfg.freq_dim))
    c = F.linear(F.silu(F.linear(e, _t(mw["w_t1"]), _t(mw["b_t1"]))), _t(mw["w_t2"]), _t(mw["b_t2"]))
    m = F.linear(F.silu(c), _t(mw["w_hmod"]), _t(mw["b_hmod"]))
    ref, off = [], 0
    for r, (Fg, Hg, Wg) in enumerate(vl.grid_fhw):
        n = C * Fg * pt * Hg * ph * Wg * pw
        lat = latent[off:off + n].reshape(C, Fg * pt, Hg * ph, Wg * pw)
        tok = rearrange(lat, "c (f i) (h j) (w k) -> (f h w) (c i j k)", i=pt, j=ph, k=pw)
        x = F.linear(_t(tok), _t(mw["w_pe"]), _t(mw["b_pe"]))
        h = F.layer_norm(x, (D,), eps=cfg.ln_eps) * (1 + m[r, D:]) + m[r, :D]
        v = F.linear(h, _t(mw["w_out"]), _t(mw["b_out"])).numpy()
        vl_r = rearrange(v, "(f h w) (c i j k) -> c (f i) (h j) (w k)", f=Fg, h=Hg, w=Wg, c=C, i=pt, j=ph, k=pw)
        ref.append((lat + dt[r] * vl_r).reshape(-1))
        off += n
    _close(out, np.concatenate(ref), 1e-12, "identity blocks")


def check_step_affine_in_dt():
    """The update is linear in dt: out(dt) - latent scales with dt."""
    st = list(_model_setup(seed=41))
    latent, dt = st[4], st[6]
    d1 = _step(st) - latent
    st[6] = 2.5 * dt
    d2 = _step(st) - latent
    _close(d2, 2.5 * d1, 1e-13, "affine in dt")


def check_step_requests_independent():
    """A packed batch equals each request stepped alone (per-request t, dt, text)."""
    st = _model_setup(seed=51)
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = st
    out = _step(st)
    sizes = M.latent_sizes(C, vl.grid_fhw, patch)
    off = 0
    for r in range(vl.n_req):
        n = vl.cu_seqlens[r + 1] - vl.cu_seqlens[r]
        lt = vl.cu_txt[r + 1] - vl.cu_txt[r]
        vr = O.Varlen([0, n], [0, lt], [vl.grid_fhw[r]])
        o_r = M.denoise_step(cfg, vr, C, patch, latent[off:off + sizes[r]], t[r:r + 1], dt[r:r + 1],
                             txt[vl.cu_txt[r]:vl.cu_txt[r + 1]], mw, blocks)
        _close(out[off:off + sizes[r]], o_r, 1e-12, f"request {r} alone")
        off += sizes[r]


def check_step_blocks_are_dit_blocks():
    """With every block's own timestep MLP set to the shared one, the step's
    velocity equals patch embedding -> block_forward (each block conditioning
    itself) -> final layer."""
    st = _model_setup(seed=61)
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = st
    _, v = _step(st, return_velocity=True)
    x = O.linear(M.patchify_packed(latent, C, vl.grid_fhw, patch), mw["w_pe"], mw["b_pe"])
    for w in blocks:
        w2 = dict(w, w_t1=mw["w_t1"], b_t1=mw["b_t1"], w_t2=mw["w_t2"], b_t2=mw["b_t2"])
        x = O.block_forward(cfg, vl, x, t, txt, w2)
    req = np.repeat(np.arange(vl.n_req), np.diff(vl.cu_seqlens))
    c = O.timestep_mlp(O.timestep_embedding(t, cfg.freq_dim), mw["w_t1"], mw["b_t1"], mw["w_t2"], mw["b_t2"])
    _close(v, M.final_layer(x, c, req, cfg.ln_eps, mw), 1e-12, "blocks inside the step")


def check_text_kv_is_cross_kv():
    """The cached text keys/values of block b are [RMS(ck) | cv] of that block."""
    st = _model_setup(seed=71)
    cfg, vl, C, patch, latent, t, dt, txt, mw, blocks = st
    kv = M.text_kv(cfg, txt, blocks)
    D, d = cfg.hidden, cfg.head_dim
    for b, w in enumerate(blocks):
        z = F.linear(_t(txt), _t(w["w_ckv"]), _t(w["b_ckv"]))
        ck = z[:, :D].reshape(-1, cfg.n_heads, d)
        ck = ck / torch.sqrt((ck * ck).mean(-1, keepdim=True) + cfg.rms_eps) * _t(w["g_ck"])
        _close(kv[b], torch.cat([ck.reshape(-1, D), z[:, D:]], 1).numpy(), 1e-12, f"text kv of block {b}")


ALL_CHECKS = [
    check_patchify_bruteforce, check_patchify_einops, check_patch_embedding_conv3d, check_patch_roundtrip,
    check_euler_on_flow_path, check_final_layer_torch, check_step_dt_zero, check_step_zero_output_weights,
    check_step_identity_blocks, check_step_affine_in_dt, check_step_requests_independent,
    check_step_blocks_are_dit_blocks, check_text_kv_is_cross_kv,
]
