"""Pins of the CPU oracle: checks against facts the oracle does not compute
itself (brute-force loops, closed forms of special cases, invariants and
independent library routines).  Each ``check_*`` raises AssertionError on a
mismatch; ``test_oracle_pins.py`` runs them on the oracle as written and
``test_oracle_mutants.py`` runs them on deliberately broken copies of it.

Every oracle call goes through the module object so that a mutant patched
into ``oracle.dit_block`` is seen by the block's internal calls too.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle import dit_block as O
import synth.gen as SG

RNG = np.random.default_rng(20260613)


def _close(a, b, tol=1e-10, what=""):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


# ---------------------------------------------------------------- timestep


def check_timestep_zero():
    """t = 0: the cosine half is 1 and the sine half is 0."""
    e = O.timestep_embedding(np.array([0.0]), 16)
    _close(e[0, :8], np.ones(8), 0, "cos half at t=0")
    _close(e[0, 8:], np.zeros(8), 0, "sin half at t=0")


def check_timestep_frequencies():
    """Frequencies are 1, r, r^2, ... with r = 10^(-4/half): recovered from the
    sine half at a tiny t (sin x ~ x), never from the oracle's own formula."""
    half = 12
    t = 1e-7
    e = O.timestep_embedding(np.array([t]), 2 * half)
    w = e[0, half:] / t
    _close(w[0], 1.0, 1e-9, "first frequency")
    _close(w[1:] / w[:-1], np.full(half - 1, 10.0 ** (-4.0 / half)), 1e-9, "frequency ratio")
    # unit circle per frequency, any t
    e = O.timestep_embedding(np.array([0.3, 17.0, 999.9]), 2 * half)
    _close(e[:, :half] ** 2 + e[:, half:] ** 2, np.ones((3, half)), 1e-12, "cos^2+sin^2")
    # first component is cos(t) exactly (frequency 1)
    _close(e[:, 0], np.cos([0.3, 17.0, 999.9]), 1e-12, "cos(t) at frequency 1")


# ---------------------------------------------------------------- activations


def check_silu():
    z = RNG.standard_normal(64) * 4
    _close(O.silu(z), F.silu(_t(z)).numpy(), 1e-13, "silu vs torch")
    _close(O.silu(z) - O.silu(-z), z, 1e-12, "silu(z)-silu(-z)=z")


def check_gelu_tanh():
    z = RNG.standard_normal(256) * 3
    _close(O.gelu_tanh(z), F.gelu(_t(z), approximate="tanh").numpy(), 1e-13, "gelu_tanh vs torch")
    _close(O.gelu_tanh(z) - O.gelu_tanh(-z), z, 1e-12, "gelu(z)-gelu(-z)=z")
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0
    # the tanh form approximates the erf form closely but not exactly
    erf = 0.5 * z * (1 + np.array([math.erf(v / math.sqrt(2)) for v in z]))
    d = np.abs(O.gelu_tanh(z) - erf).max()
    assert 0 < d < 1e-3, f"tanh-GELU vs erf-GELU {d}"


# ---------------------------------------------------------------- linear


def check_linear_bruteforce():
    m, k, n = 3, 5, 4
    z = RNG.standard_normal((m, k))
    w = RNG.standard_normal((n, k))
    b = RNG.standard_normal(n)
    ref = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            s = b[j]
            for kk in range(k):
                s += z[i, kk] * w[j, kk]
            ref[i, j] = s
    _close(O.linear(z, w, b), ref, 1e-12, "linear vs loops")
    _close(O.linear(z, w, b), F.linear(_t(z), _t(w), _t(b)).numpy(), 1e-12, "linear vs torch")


# ---------------------------------------------------------------- norms


def check_layer_norm():
    z = RNG.standard_normal((7, 48)) * 3 + 1.5
    eps = 1e-6
    out = O.layer_norm(z, eps)
    _close(out, F.layer_norm(_t(z), (48,), eps=eps).numpy(), 1e-12, "layer_norm vs torch")
    _close(out.mean(axis=1), np.zeros(7), 1e-12, "row mean 0")
    var = z.var(axis=1)
    _close(out.var(axis=1), var / (var + eps), 1e-12, "row variance s2/(s2+eps)")
    # large eps makes the biased-variance choice visible
    _close(O.layer_norm(z, 0.5), F.layer_norm(_t(z), (48,), eps=0.5).numpy(), 1e-12, "eps=0.5")


def check_modulate():
    hn = RNG.standard_normal((4, 8))
    sh, sc = RNG.standard_normal(8), RNG.standard_normal(8)
    _close(O.modulate(hn, np.zeros(8), np.zeros(8)), hn, 0, "scale=shift=0 is identity")
    _close(O.modulate(hn, sh, -np.ones(8)), np.broadcast_to(sh, hn.shape), 0, "scale=-1 gives shift")
    _close(O.modulate(hn, sh, sc) - O.modulate(hn, sh, np.zeros(8)), hn * sc, 1e-12, "linear in scale")


def check_rms_norm_heads():
    H, d, eps = 3, 8, 1e-6
    u = RNG.standard_normal((5, H * d)) * 2
    g = 1 + 0.1 * RNG.standard_normal(d)
    out = O.rms_norm_heads(u, g, H, d, eps)
    ref = F.rms_norm(_t(u.reshape(5, H, d)), (d,), weight=_t(g), eps=eps).numpy().reshape(5, H * d)
    _close(out, ref, 1e-12, "rms_norm vs torch")
    # rms(out / g) = sqrt(m / (m + eps)) per head
    v = (out.reshape(5, H, d) / g)
    m = (u.reshape(5, H, d) ** 2).mean(-1)
    _close(np.sqrt((v ** 2).mean(-1)), np.sqrt(m / (m + eps)), 1e-12, "rms after norm")
    # heads are independent: changing head 1 leaves heads 0 and 2 alone
    u2 = u.copy()
    u2[:, d:2 * d] *= 7.0
    out2 = O.rms_norm_heads(u2, g, H, d, eps)
    _close(out2[:, :d], out[:, :d], 1e-14, "head 0 independent of head 1")
    _close(out2[:, 2 * d:], out[:, 2 * d:], 1e-14, "head 2 independent of head 1")


# ---------------------------------------------------------------- rotary


def check_grid_positions():
    grid = (3, 4, 5)
    ref = []
    for f in range(grid[0]):
        for h in range(grid[1]):
            for w in range(grid[2]):
                ref.append((f, h, w))
    ref = np.array(ref)
    _close(O.grid_positions(60, grid), ref, 0, "row-major (t,h,w)")
    _close(O.grid_positions(17, grid, offset=23), ref[23:40], 0, "offset")


def _rope1d_complex(u, pos, d, theta):
    """Standard 1D RoPE written with complex numbers: pair j is the complex
    number u[2j] + i u[2j+1], multiplied by exp(i p theta^(-2j/d))."""
    z = u[..., 0::2] + 1j * u[..., 1::2]
    j = np.arange(d // 2)
    rot = np.exp(1j * pos[:, None] * theta ** (-2.0 * j / d))
    zr = z * rot
    out = np.empty_like(u)
    out[..., 0::2] = zr.real
    out[..., 1::2] = zr.imag
    return out


def check_rope():
    n, H, d, theta = 6, 2, 16, 10000.0
    u = RNG.standard_normal((n, H * d))
    # one section covering the head == standard 1D RoPE (complex form)
    pos = np.stack([np.zeros(n, int), np.arange(n) * 3 + 1, np.zeros(n, int)], 1)
    ang = O.rope_angles(pos, (0, d, 0), theta)
    out = O.apply_rope(u, H, d, ang)
    ref = np.concatenate([_rope1d_complex(u[:, h * d:(h + 1) * d], pos[:, 1].astype(float), d, theta)
                          for h in range(H)], axis=1)
    _close(out, ref, 1e-12, "single section == 1D RoPE")
    # sectioned: each section is 1D RoPE on its own slice with its own axis
    sec = (4, 6, 6)
    pos = np.stack([RNG.integers(0, 9, n), RNG.integers(0, 30, n), RNG.integers(0, 50, n)], 1)
    out = O.apply_rope(u, H, d, O.rope_angles(pos, sec, theta))
    a = 0
    for s, ds in enumerate(sec):
        for h in range(H):
            sl = slice(h * d + a, h * d + a + ds)
            _close(out[:, sl], _rope1d_complex(u[:, sl], pos[:, s].astype(float), ds, theta),
                   1e-12, f"section {s}")
        a += ds
    # norm of every pair preserved
    pr = out.reshape(n, -1, 2)
    pu = u.reshape(n, -1, 2)
    _close((pr ** 2).sum(-1), (pu ** 2).sum(-1), 1e-12, "pair norms")
    # position 0 is the identity
    _close(O.apply_rope(u, H, d, O.rope_angles(np.zeros((n, 3), int), sec, theta)), u, 0, "pos 0")
    # relative property: <R_p q, R_p' k> depends on p' - p only (per axis)
    q = RNG.standard_normal((1, d))
    k = RNG.standard_normal((1, d))
    def dot(p, pp):
        rq = O.apply_rope(q, 1, d, O.rope_angles(np.array([p]), sec, theta))
        rk = O.apply_rope(k, 1, d, O.rope_angles(np.array([pp]), sec, theta))
        return float((rq * rk).sum())
    _close(dot((1, 5, 9), (3, 2, 20)), dot((0, 0, 0), (2, -3, 11)), 1e-11, "relative position")


# ---------------------------------------------------------------- attention


def check_attention_bruteforce():
    nq, nk, d = 4, 6, 5
    q, k, v = RNG.standard_normal((nq, d)), RNG.standard_normal((nk, d)), RNG.standard_normal((nk, 3))
    sc = 0.37
    ref = np.zeros((nq, 3))
    for i in range(nq):
        logits = [sum(q[i, c] * k[j, c] for c in range(d)) * sc for j in range(nk)]
        mx = max(logits)
        ex = [math.exp(l - mx) for l in logits]
        tot = sum(ex)
        for c in range(3):
            ref[i, c] = sum(ex[j] / tot * v[j, c] for j in range(nk))
    _close(O.attention(q, k, v, sc), ref, 1e-12, "attention vs loops")
    # vs torch SDPA (float64, CPU), default scale 1/sqrt(d)
    H, dd, n = 3, 8, 9
    Q, K, V = (RNG.standard_normal((n, H * dd)) for _ in range(3))
    out = O.attention_varlen(Q, K, V, [0, n], [0, n], H, dd)
    tq = _t(Q.reshape(n, H, dd).transpose(1, 0, 2))
    tk = _t(K.reshape(n, H, dd).transpose(1, 0, 2))
    tv = _t(V.reshape(n, H, dd).transpose(1, 0, 2))
    ref = F.scaled_dot_product_attention(tq, tk, tv).numpy().transpose(1, 0, 2).reshape(n, H * dd)
    _close(out, ref, 1e-12, "attention vs torch sdpa")


def check_attention_invariants():
    nq, nk, d = 5, 7, 4
    q, k = RNG.standard_normal((nq, d)), RNG.standard_normal((nk, d))
    # V = identity exposes the probabilities: rows sum to one, all positive
    p = O.attention(q, k, np.eye(nk), 0.5)
    _close(p.sum(1), np.ones(nq), 1e-13, "rows of P sum to 1")
    assert (p > 0).all()
    v = RNG.standard_normal((nk, 3))
    # a single key gives its value
    _close(O.attention(q, k[:1], v[:1], 0.5), np.repeat(v[:1], nq, 0), 1e-14, "single key")
    # identical keys give the mean of the values
    _close(O.attention(q, np.repeat(k[:1], nk, 0), v, 0.5), np.repeat(v.mean(0, keepdims=True), nq, 0),
           1e-13, "identical keys")
    # a constant added to every logit of a row (via an extra dimension) changes nothing
    q2 = np.concatenate([q, np.ones((nq, 1))], 1)
    k2 = np.concatenate([k, np.full((nk, 1), 3.0)], 1)
    _close(O.attention(q2, k2, v, 0.5), O.attention(q, k, v, 0.5), 1e-12, "logit shift")


def check_attention_varlen():
    H, d = 2, 4
    cu_q, cu_k = [0, 3, 3, 8], [0, 2, 5, 9]
    Q = RNG.standard_normal((8, H * d))
    K = RNG.standard_normal((9, H * d))
    V = RNG.standard_normal((9, H * d))
    out = O.attention_varlen(Q, K, V, cu_q, cu_k, H, d)
    for r in range(3):
        if cu_q[r] == cu_q[r + 1]:
            continue
        one = O.attention_varlen(Q[cu_q[r]:cu_q[r + 1]], K[cu_k[r]:cu_k[r + 1]], V[cu_k[r]:cu_k[r + 1]],
                                 [0, cu_q[r + 1] - cu_q[r]], [0, cu_k[r + 1] - cu_k[r]], H, d)
        _close(out[cu_q[r]:cu_q[r + 1]], one, 1e-14, f"request {r} alone")
    # sampled query rows equal the full computation's rows
    rows = np.array([0, 4, 7])
    _close(O.attention_varlen(Q, K, V, cu_q, cu_k, H, d, q_rows=rows), out[rows], 1e-14, "q_rows")


# ---------------------------------------------------------------- block


def tiny_setup(seed=1, R=2, rows=(3, 4), L=3, D=8, H=2, Dff=16, sections=(0, 2, 2),
               grids=((1, 2, 2), (1, 2, 3))):
    rng = np.random.default_rng(seed)
    d = D // H
    cfg = O.BlockConfig(hidden=D, n_heads=H, head_dim=d, mlp_hidden=Dff, freq_dim=D,
                        rope_sections=tuple(sections))
    cu = [0]
    for r in rows:
        cu.append(cu[-1] + r)
    vl = O.Varlen(cu_seqlens=cu, cu_txt=[i * L for i in range(R + 1)], grid_fhw=list(grids))
    s = 0.3
    w = {
        "w_t1": rng.standard_normal((D, D)) * s, "b_t1": rng.standard_normal(D) * s,
        "w_t2": rng.standard_normal((D, D)) * s, "b_t2": rng.standard_normal(D) * s,
        "w_ada": rng.standard_normal((6 * D, D)) * s, "b_ada": rng.standard_normal(6 * D) * s,
        "w_qkv": rng.standard_normal((3 * D, D)) * s, "b_qkv": rng.standard_normal(3 * D) * s,
        "g_q": 1 + 0.2 * rng.standard_normal(d), "g_k": 1 + 0.2 * rng.standard_normal(d),
        "w_o": rng.standard_normal((D, D)) * s, "b_o": rng.standard_normal(D) * s,
        "g_ca": 1 + 0.2 * rng.standard_normal(D), "b_ca": 0.2 * rng.standard_normal(D),
        "w_cq": rng.standard_normal((D, D)) * s, "b_cq": rng.standard_normal(D) * s,
        "w_ckv": rng.standard_normal((2 * D, D)) * s, "b_ckv": rng.standard_normal(2 * D) * s,
        "g_cq": 1 + 0.2 * rng.standard_normal(d), "g_ck": 1 + 0.2 * rng.standard_normal(d),
        "w_co": rng.standard_normal((D, D)) * s, "b_co": rng.standard_normal(D) * s,
        "w_up": rng.standard_normal((Dff, D)) * s, "b_up": rng.standard_normal(Dff) * s,
        "w_dn": rng.standard_normal((D, Dff)) * s, "b_dn": rng.standard_normal(D) * s,
    }
    x = rng.standard_normal((cu[-1], D))
    txt = rng.standard_normal((R * L, D))
    t = rng.uniform(0, 1000, R)
    return cfg, vl, x, t, txt, w


def _req_of_rows(vl):
    return np.concatenate([np.full(vl.cu_seqlens[r + 1] - vl.cu_seqlens[r], r) for r in range(vl.n_req)])


def check_block_identity():
    """Zero adaLN gates and a zero cross-attention output projection give y = x
    exactly (the cross residual is ungated, so it has to be zeroed too)."""
    cfg, vl, x, t, txt, w = tiny_setup()
    D = cfg.hidden
    w["w_ada"][2 * D:3 * D] = 0
    w["b_ada"][2 * D:3 * D] = 0
    w["w_ada"][5 * D:6 * D] = 0
    w["b_ada"][5 * D:6 * D] = 0
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    y = O.block_forward(cfg, vl, x, t, txt, w)
    assert np.array_equal(y, x), "zero gates must give the identity"


def _zero_ada(w, D, chunks):
    w["w_ada"][:] = 0
    for c, val in chunks.items():
        w["b_ada"][c * D:(c + 1) * D] = val


def check_block_self_branch_closed_form():
    """W_qkv = 0: q, k, v are the biases for every row, the softmax is uniform
    and the attention output is b_v; with W_ada = 0 the gates are chunks of
    b_ada, so y - x = gate_sa * (W_o b_v + b_o) when the other branches are off."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=2, sections=(0, 0, 0))
    D = cfg.hidden
    rng = np.random.default_rng(5)
    gate = rng.standard_normal(D)
    _zero_ada(w, D, {2: gate, 5: 0.0, 0: rng.standard_normal(D), 1: rng.standard_normal(D)})
    w["w_qkv"][:] = 0
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    b_v = w["b_qkv"][2 * D:]
    proj = np.array([sum(w["w_o"][i, j] * b_v[j] for j in range(D)) + w["b_o"][i] for i in range(D)])
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, np.broadcast_to(gate * proj, x.shape), 1e-12, "self branch closed form")


def check_block_cross_branch_closed_form():
    """W_ckv = 0: text keys and values are constant per request, so the cross
    output is b_cv and y - x = W_co b_cv + b_co (ungated) with both gates 0."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=3)
    D = cfg.hidden
    _zero_ada(w, D, {2: 0.0, 5: 0.0})
    w["w_ckv"][:] = 0
    b_cv = w["b_ckv"][D:]
    proj = np.array([sum(w["w_co"][i, j] * b_cv[j] for j in range(D)) + w["b_co"][i] for i in range(D)])
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, np.broadcast_to(proj, x.shape), 1e-12, "cross branch closed form")


def check_block_mlp_branch_closed_form():
    """W_up = 0: the MLP hidden is gelu_tanh(b_up) for every row, so
    y - x = gate_ff * (W_dn gelu(b_up) + b_dn) with the attention gate and the
    cross output projection at zero."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=4)
    D = cfg.hidden
    rng = np.random.default_rng(6)
    gate = rng.standard_normal(D)
    _zero_ada(w, D, {2: 0.0, 5: gate})
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    w["w_up"][:] = 0
    g = F.gelu(_t(w["b_up"]), approximate="tanh").numpy()
    proj = np.array([sum(w["w_dn"][i, j] * g[j] for j in range(cfg.mlp_hidden)) + w["b_dn"][i]
                     for i in range(D)])
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, np.broadcast_to(gate * proj, x.shape), 1e-12, "mlp branch closed form")


def check_block_attn_modulation_closed_form():
    """q and k constant (W_q = W_k = 0) make self-attention a per-request mean;
    with W_v = W_o = I and zero biases, y - x = gate_sa * mean_req(LN(x)(1+scale_sa)+shift_sa).
    LayerNorm from torch."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=7, sections=(0, 0, 0))
    D = cfg.hidden
    rng = np.random.default_rng(8)
    shift, scale, gate = (rng.standard_normal(D) for _ in range(3))
    _zero_ada(w, D, {0: shift, 1: scale, 2: gate, 5: 0.0})
    w["w_qkv"][:2 * D] = 0
    w["w_qkv"][2 * D:] = np.eye(D)
    w["b_qkv"][2 * D:] = 0
    w["w_o"][:] = np.eye(D)
    w["b_o"][:] = 0
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    h = F.layer_norm(_t(x), (D,), eps=cfg.ln_eps).numpy() * (1 + scale) + shift
    exp = np.empty_like(x)
    for r in range(vl.n_req):
        a, b = vl.cu_seqlens[r], vl.cu_seqlens[r + 1]
        exp[a:b] = gate * h[a:b].mean(0)
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, exp, 1e-12, "attention-input modulation closed form")


def check_block_mlp_modulation_closed_form():
    """With Dff = D, W_up = W_dn = I and zero biases, and the other branches
    off, y - x = gate_ff * gelu_tanh(LN(x)(1+scale_ff)+shift_ff) (torch ops)."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=9, Dff=8)
    D = cfg.hidden
    rng = np.random.default_rng(10)
    shift, scale, gate = (rng.standard_normal(D) for _ in range(3))
    _zero_ada(w, D, {2: 0.0, 3: shift, 4: scale, 5: gate})
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    w["w_up"][:] = np.eye(D)
    w["b_up"][:] = 0
    w["w_dn"][:] = np.eye(D)
    w["b_dn"][:] = 0
    h = F.layer_norm(_t(x), (D,), eps=cfg.ln_eps) * _t(1 + scale) + _t(shift)
    exp = gate * F.gelu(h, approximate="tanh").numpy()
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, exp, 1e-12, "mlp-input modulation closed form")


def _torch_rope(u, pos, sections, theta, H, d):
    """Sectioned RoPE via complex multiplication (independent of the oracle)."""
    out = u.copy()
    for h in range(H):
        a = 0
        for s, ds in enumerate(sections):
            if ds:
                sl = slice(h * d + a, h * d + a + ds)
                out[:, sl] = _rope1d_complex(u[:, sl], pos[:, s].astype(float), ds, theta)
            a += ds
    return out


def check_block_cross_attention_torch():
    """Both gates 0 and W_co = I, b_co = 0: y - x is the cross-attention output,
    rebuilt from torch layer_norm, rms_norm and scaled_dot_product_attention
    per request (text rows cu_txt[r]..cu_txt[r+1])."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=11)
    D, H, d = cfg.hidden, cfg.n_heads, cfg.head_dim
    _zero_ada(w, D, {2: 0.0, 5: 0.0})
    w["w_co"][:] = np.eye(D)
    w["b_co"][:] = 0
    hc = F.layer_norm(_t(x), (D,), weight=_t(w["g_ca"]), bias=_t(w["b_ca"]), eps=cfg.ln_eps)
    cq = F.linear(hc, _t(w["w_cq"]), _t(w["b_cq"])).reshape(-1, H, d)
    cq = F.rms_norm(cq, (d,), weight=_t(w["g_cq"]), eps=cfg.rms_eps)
    ckv = F.linear(_t(txt), _t(w["w_ckv"]), _t(w["b_ckv"]))
    ck = F.rms_norm(ckv[:, :D].reshape(-1, H, d), (d,), weight=_t(w["g_ck"]), eps=cfg.rms_eps)
    cv = ckv[:, D:].reshape(-1, H, d)
    exp = np.empty_like(x)
    for r in range(vl.n_req):
        a, b = vl.cu_seqlens[r], vl.cu_seqlens[r + 1]
        ta, tb = vl.cu_txt[r], vl.cu_txt[r + 1]
        o = F.scaled_dot_product_attention(cq[a:b].transpose(0, 1), ck[ta:tb].transpose(0, 1),
                                           cv[ta:tb].transpose(0, 1))
        exp[a:b] = o.transpose(0, 1).reshape(b - a, D).numpy()
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, exp, 1e-12, "cross attention vs torch")


def check_block_self_attention_torch():
    """Only the self-attention branch on (W_ada = 0, gate_sa from b_ada, cross
    output projection and gate_ff zero): y - x = gate_sa * (SDPA(rope(rms(q)),
    rope(rms(k)), v) W_o^T + b_o), rebuilt from torch ops and a complex-number
    rotary per request grid."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=12, rows=(4, 6), grids=((1, 2, 2), (2, 1, 3)))
    D, H, d = cfg.hidden, cfg.n_heads, cfg.head_dim
    rng = np.random.default_rng(13)
    shift, scale, gate = (rng.standard_normal(D) for _ in range(3))
    _zero_ada(w, D, {0: shift, 1: scale, 2: gate, 5: 0.0})
    w["w_co"][:] = 0
    w["b_co"][:] = 0
    h = F.layer_norm(_t(x), (D,), eps=cfg.ln_eps) * _t(1 + scale) + _t(shift)
    qkv = F.linear(h, _t(w["w_qkv"]), _t(w["b_qkv"])).numpy()
    q = F.rms_norm(_t(qkv[:, :D].reshape(-1, H, d)), (d,), weight=_t(w["g_q"]), eps=cfg.rms_eps)
    k = F.rms_norm(_t(qkv[:, D:2 * D].reshape(-1, H, d)), (d,), weight=_t(w["g_k"]), eps=cfg.rms_eps)
    q = q.reshape(-1, D).numpy()
    k = k.reshape(-1, D).numpy()
    v = qkv[:, 2 * D:]
    o = np.empty_like(x)
    for r in range(vl.n_req):
        a, b = vl.cu_seqlens[r], vl.cu_seqlens[r + 1]
        Fg, Hg, Wg = vl.grid_fhw[r]
        pos = np.array([(g // (Hg * Wg), (g // Wg) % Hg, g % Wg) for g in range(b - a)])
        qr = _torch_rope(q[a:b], pos, cfg.rope_sections, cfg.rope_theta, H, d)
        kr = _torch_rope(k[a:b], pos, cfg.rope_sections, cfg.rope_theta, H, d)
        oo = F.scaled_dot_product_attention(_t(qr.reshape(-1, H, d)).transpose(0, 1),
                                            _t(kr.reshape(-1, H, d)).transpose(0, 1),
                                            _t(v[a:b].reshape(-1, H, d)).transpose(0, 1))
        o[a:b] = oo.transpose(0, 1).reshape(b - a, D).numpy()
    exp = gate * F.linear(_t(o), _t(w["w_o"]), _t(w["b_o"])).numpy()
    y = O.block_forward(cfg, vl, x, t, txt, w)
    _close(y - x, exp, 1e-12, "self attention vs torch")


def check_block_conditioning_torch():
    """S0 rebuilt from torch: sinusoid (cos, sin; frequencies 10^(-4 i/half)),
    Linear-SiLU-Linear, SiLU, Linear(D -> 6D)."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=14)
    half = cfg.freq_dim // 2
    fr = torch.tensor([10.0 ** (-4.0 * i / half) for i in range(half)], dtype=torch.float64)
    arg = _t(t)[:, None] * fr[None]
    e = torch.cat([torch.cos(arg), torch.sin(arg)], 1)
    c = F.linear(F.silu(F.linear(e, _t(w["w_t1"]), _t(w["b_t1"]))), _t(w["w_t2"]), _t(w["b_t2"]))
    m = F.linear(F.silu(c), _t(w["w_ada"]), _t(w["b_ada"])).numpy().reshape(len(t), 6, -1)
    _close(O.conditioning(t, cfg.freq_dim, w), m, 1e-12, "conditioning vs torch")


def check_block_permutation_equivariance():
    """Without rotary, permuting a request's rows permutes its outputs."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=15, sections=(0, 0, 0), rows=(4, 5))
    perm = np.concatenate([np.array([2, 0, 3, 1]), 4 + np.array([4, 1, 0, 3, 2])])
    y = O.block_forward(cfg, vl, x, t, txt, w)
    yp = O.block_forward(cfg, vl, x[perm], t, txt, w)
    _close(yp, y[perm], 1e-12, "permutation equivariance")


def check_block_composition_and_rows():
    """pre -> attention -> post equals block_forward; the sampled-row mode
    equals the full output rows; a shard with a position offset equals the
    corresponding rows of the full request's pre-attention outputs."""
    cfg, vl, x, t, txt, w = tiny_setup(seed=16, rows=(4, 6), grids=((1, 2, 2), (2, 1, 3)))
    mod = O.conditioning(t, cfg.freq_dim, w)
    y = O.block_forward(cfg, vl, x, t, txt, w)
    q, k, v = O.pre_attention(cfg, vl, x, w, mod)
    o = O.attention_varlen(q, k, v, vl.cu_seqlens, vl.cu_seqlens, cfg.n_heads, cfg.head_dim)
    _close(O.post_attention(cfg, vl, x, o, txt, w, mod), y, 1e-14, "composition")
    rows = np.array([0, 3, 4, 8, 9])
    _close(O.block_forward_rows(cfg, vl, x, t, txt, w, rows, row_chunk=3), y[rows], 1e-12, "rows mode")
    # shard: rows 2..5 of request 1 with pos_offset 2 == rows 2..5 of the full request
    sub = O.Varlen([0, 3], [0, 3], [vl.grid_fhw[1]], pos_offset=[2])
    qs, ks, vs = O.pre_attention(cfg, sub, x[6:9], w, mod[1:2])
    _close(qs, q[6:9], 1e-14, "shard q")
    _close(ks, k[6:9], 1e-14, "shard k")


# ---------------------------------------------------------------- bf16 storage


def _bits(words):
    return np.array(words, dtype=np.uint16)


def _f32(words):
    return np.array(words, dtype=np.uint32).view(np.float32)


def check_bf16_codec():
    """The stored-value decoding every parity check reads through (oracle
    ``decode``) and the encoder that writes the bf16 inputs both sides read
    (``synth.gen.bf16_bits``).  bfloat16 is the top half of an IEEE binary32
    word: sign, 8 exponent bits (bias 127), 7 mantissa bits; the encoder
    rounds to nearest, ties to even.  Checked on hand-worked bit patterns and
    against torch's own float32 -> bfloat16 conversion."""
    # decode: hand-worked patterns
    words = [0x3F80, 0xBF80, 0x4049, 0x3C00, 0x0000, 0x0001, 0x007F, 0x0080, 0x7F7F, 0x7F80, 0xFF80, 0xC2F7]
    want = [1.0, -1.0, 3.140625, 2.0 ** -7, 0.0, 2.0 ** -133, 127 * 2.0 ** -133, 2.0 ** -126,
            (2 - 2.0 ** -7) * 2.0 ** 127, math.inf, -math.inf, -123.5]
    got = O.decode(_bits(words))
    assert got.dtype == np.float64, f"decode gives {got.dtype}"
    for wd, g, v in zip(words, got, want):
        assert g == v, f"decode(0x{wd:04X}) = {g!r}, expected {v!r}"
    neg0 = O.decode(_bits([0x8000]))[0]
    assert neg0 == 0.0 and math.copysign(1.0, neg0) < 0, "decode(0x8000) is not -0.0"
    # float32 storage decodes to itself
    f = np.array([1.5, -2.25e-30, 3.0e38], dtype=np.float32)
    assert np.array_equal(O.decode(f), f.astype(np.float64)), "float32 decode"
    # encode: hand-worked round-to-nearest-even cases (float32 word -> bf16 word)
    cases = [
        (0x3F800000, 0x3F80),   # 1.0
        (0x3F808000, 0x3F80),   # 1 + 2^-8: a tie, 0x3F80 is even
        (0x3F818000, 0x3F82),   # 1 + 3*2^-8: a tie, 0x3F81 is odd -> up
        (0x3F808001, 0x3F81),   # just above the tie
        (0x3F807FFF, 0x3F80),   # just below the tie
        (0xBF818000, 0xBF82),   # the odd tie, negative
        (0x00010000, 0x0001),   # smallest bf16 subnormal
        (0x00018000, 0x0002),   # subnormal tie -> even
        (0x00008000, 0x0000),   # half the smallest subnormal: tie -> +0
        (0x7F7FFFFF, 0x7F80),   # float32 max rounds past bf16 max to inf
        (0x7F7F7FFF, 0x7F7F),   # stays at bf16 max
        (0x80000000, 0x8000),   # -0.0
        (0x7F800000, 0x7F80),   # inf
    ]
    enc = SG.bf16_bits(_f32([c[0] for c in cases]))
    assert enc.dtype == np.uint16, f"bf16_bits gives {enc.dtype}"
    for (src, dst), e in zip(cases, enc):
        assert int(e) == dst, f"bf16_bits(0x{src:08X}) = 0x{int(e):04X}, expected 0x{dst:04X}"
    # against torch's conversion: random magnitudes from 2^-140 to 2^120, both
    # signs, with every other value forced onto an exact tie (low half 0x8000)
    rng = np.random.default_rng(7)
    n = 4096
    x = (rng.standard_normal(n) * np.exp2(rng.integers(-140, 120, n))).astype(np.float32)
    u = x.view(np.uint32).copy()
    u[::2] = (u[::2] & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    u[1::4] |= np.uint32(0x00010000)    # odd bf16 LSB under some of the ties
    x = u.view(np.float32)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16)
    ref_bits = ref.view(torch.int16).numpy().view(np.uint16)
    enc = SG.bf16_bits(x)
    bad = np.nonzero(enc != ref_bits)[0]
    assert bad.size == 0, f"bf16_bits differs from torch at {bad.size} values, e.g. 0x{u[bad[0]]:08X}"
    assert np.array_equal(O.decode(ref_bits), ref.double().numpy()), "decode differs from torch bfloat16 -> float64"
    # the round trip lands within half a bf16 unit (2^-8 relative) of the source
    rt = O.decode(SG.bf16_bits(x))
    fin = np.isfinite(rt) & (np.abs(x) >= 2.0 ** -126)
    rel = np.abs(rt[fin] - x[fin]) / np.abs(x[fin].astype(np.float64))
    assert rel.max() <= 2.0 ** -8, f"round trip relative error {rel.max():.3e}"


ALL_CHECKS = [
    check_bf16_codec,
    check_timestep_zero, check_timestep_frequencies, check_silu, check_gelu_tanh,
    check_linear_bruteforce, check_layer_norm, check_modulate, check_rms_norm_heads,
    check_grid_positions, check_rope, check_attention_bruteforce, check_attention_invariants,
    check_attention_varlen, check_block_identity, check_block_self_branch_closed_form,
    check_block_cross_branch_closed_form, check_block_mlp_branch_closed_form,
    check_block_attn_modulation_closed_form, check_block_mlp_modulation_closed_form,
    check_block_cross_attention_torch, check_block_self_attention_torch,
    check_block_conditioning_torch, check_block_permutation_equivariance,
    check_block_composition_and_rows,
]
