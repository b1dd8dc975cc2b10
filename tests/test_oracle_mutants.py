"""Plant plausible mistakes in the oracle (on the CPU) and require that at
least one pin catches each.  This is what makes the pins worth trusting: a
dropped term, a wrong sign or index or a transposed operand must not pass."""
import numpy as np
import pytest

from oracle import dit_block as O
import synth.gen as SG
from oracle_pins import ALL_CHECKS


def _fails(checks):
    failed = []
    for c in checks:
        try:
            c()
        except AssertionError:
            failed.append(c.__name__)
    return failed


orig = {n: getattr(O, n) for n in dir(O) if callable(getattr(O, n))}


def m_ln_unbiased(z, eps):
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).sum(axis=-1, keepdims=True) / (z.shape[-1] - 1)
    return (z - mu) / np.sqrt(var + eps)


def m_ln_eps_outside(z, eps):
    mu = z.mean(axis=-1, keepdims=True)
    return (z - mu) / (np.sqrt(((z - mu) ** 2).mean(axis=-1, keepdims=True)) + eps)


def m_modulate_no_one(hn, shift, scale):
    return hn * scale + shift


def m_timestep_sin_cos(t, freq_dim, max_period=10000.0):
    e = orig["timestep_embedding"](t, freq_dim, max_period)
    h = freq_dim // 2
    return np.concatenate([e[:, h:], e[:, :h]], axis=1)


def m_timestep_freq(t, freq_dim, max_period=10000.0):
    t = np.asarray(t, dtype=np.float64).reshape(-1)
    half = freq_dim // 2
    w = np.exp(-np.log(max_period) * np.arange(half) / (half - 1))
    a = t[:, None] * w[None]
    return np.concatenate([np.cos(a), np.sin(a)], 1)


def m_ada_order(c, w_ada, b_ada):
    m = orig["adaln_modulation"](c, w_ada, b_ada)
    return m[:, [0, 2, 1, 3, 5, 4]]


def m_rms_full_width(u, gamma, n_heads, head_dim, eps):
    ms = (u * u).mean(axis=-1, keepdims=True)
    return (u / np.sqrt(ms + eps)).reshape(u.shape[0], n_heads, head_dim).__mul__(gamma).reshape(u.shape)


def m_rope_half_split(u, n_heads, head_dim, angles):
    n = u.shape[0]
    v = u.reshape(n, n_heads, head_dim)
    a, b = v[..., : head_dim // 2], v[..., head_dim // 2:]
    c, s = np.cos(angles)[:, None], np.sin(angles)[:, None]
    return np.concatenate([a * c - b * s, a * s + b * c], -1).reshape(n, -1)


def m_rope_sign(u, n_heads, head_dim, angles):
    return orig["apply_rope"](u, n_heads, head_dim, -angles)


def m_rope_freq(pos, sections, theta):
    cols = []
    for s, ds in enumerate(sections):
        if ds:
            j = np.arange(ds // 2)
            cols.append(pos[:, s:s + 1] * theta ** (-j / ds)[None])
    return np.concatenate(cols, 1)


def m_grid_transposed(n_rows, grid_fhw, offset=0):
    _, Hg, Wg = grid_fhw
    g = np.arange(n_rows) + offset
    return np.stack([g // (Hg * Wg), g % Hg, (g // Hg) % Wg], 1)


def m_attn_no_scale(q, k, v, scale, q_chunk=1024):
    return orig["attention"](q, k, v, 1.0, q_chunk)


def m_attn_transposed_v(q, k, v, scale, q_chunk=1024):
    s = np.matmul(q, k.T) * scale
    p = np.exp(s - s.max(1, keepdims=True))
    p /= p.sum(0, keepdims=True)
    return np.matmul(p, v)


def m_gelu_erf(z):
    from math import erf, sqrt
    return 0.5 * z * (1 + np.vectorize(lambda x: erf(x / sqrt(2)))(z))


def m_silu_sigmoid(z):
    return 1 / (1 + np.exp(-z))


def m_linear_no_bias(z, w, b):
    return np.matmul(z, w.T)


def m_post_gated_cross(cfg, vl, x, o, txt, w, mod):
    # cross residual gated by gate_sa
    D = cfg.hidden
    req = O._row_request(vl, x.shape[0])
    w2 = dict(w)
    y = orig["post_attention"](cfg, vl, x, o, txt, w, mod)
    w2["w_co"] = np.zeros_like(w["w_co"])
    w2["b_co"] = np.zeros_like(w["b_co"])
    y0 = orig["post_attention"](cfg, vl, x, o, txt, w2, mod)
    return y0 + (y - y0) * mod[req, 2]


def m_post_no_affine(cfg, vl, x, o, txt, w, mod):
    w2 = dict(w)
    w2["g_ca"] = np.ones_like(w["g_ca"])
    w2["b_ca"] = np.zeros_like(w["b_ca"])
    return orig["post_attention"](cfg, vl, x, o, txt, w2, mod)


def m_cross_kv_swapped(cfg, txt, w):
    ck, cv = orig["cross_kv"](cfg, txt, w)
    return cv, ck


def m_pre_kv_swapped(cfg, vl, x, w, mod):
    q, k, v = orig["pre_attention"](cfg, vl, x, w, mod)
    return q, v, k


MUTANTS = {
    "layer_norm unbiased variance": ("layer_norm", m_ln_unbiased),
    "layer_norm eps outside root": ("layer_norm", m_ln_eps_outside),
    "modulate without 1+": ("modulate", m_modulate_no_one),
    "timestep sin before cos": ("timestep_embedding", m_timestep_sin_cos),
    "timestep frequency exponent i/(half-1)": ("timestep_embedding", m_timestep_freq),
    "adaLN chunk order": ("adaln_modulation", m_ada_order),
    "RMSNorm over full width": ("rms_norm_heads", m_rms_full_width),
    "rotary half-split pairs": ("apply_rope", m_rope_half_split),
    "rotary sign": ("apply_rope", m_rope_sign),
    "rotary exponent j/d": ("rope_angles", m_rope_freq),
    "grid positions transposed": ("grid_positions", m_grid_transposed),
    "attention without 1/sqrt(d)": ("attention", m_attn_no_scale),
    "softmax over the wrong axis": ("attention", m_attn_transposed_v),
    "GELU erf instead of tanh": ("gelu_tanh", m_gelu_erf),
    "SiLU as sigmoid": ("silu", m_silu_sigmoid),
    "linear drops bias": ("linear", m_linear_no_bias),
    "cross residual gated": ("post_attention", m_post_gated_cross),
    "cross LayerNorm without affine": ("post_attention", m_post_no_affine),
    "text k and v swapped": ("cross_kv", m_cross_kv_swapped),
    "self k and v swapped": ("pre_attention", m_pre_kv_swapped),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    fn_name, fn = MUTANTS[name]
    monkeypatch.setattr(O, fn_name, fn)
    failed = _fails(ALL_CHECKS)
    assert failed, f"no pin catches the mutant {name!r}"


# ------------------------------------------------ the bf16 storage format
# The oracle's decoding and the shared input encoder, each broken the way a
# plausible implementation could be.


def m_decode_shift15(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(15)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def m_decode_fp16(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return a.view(np.float16).astype(np.float64)
    return a.astype(np.float64)


def m_decode_float32_of_sign(a):
    # drops the sign bit (masks with 0x7FFF)
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return ((a.astype(np.uint32) & np.uint32(0x7FFF)) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def m_bits_half_up(a):
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x8000)) >> np.uint32(16)).astype(np.uint16)


def m_bits_truncate(a):
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def m_bits_ties_odd(a):
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + (np.uint32(1) - lsb)) >> np.uint32(16)).astype(np.uint16)


CODEC_MUTANTS = {
    "decode shifts by 15": (O, "decode", m_decode_shift15),
    "decode reads float16": (O, "decode", m_decode_fp16),
    "decode drops the sign": (O, "decode", m_decode_float32_of_sign),
    "bf16_bits rounds half up": (SG, "bf16_bits", m_bits_half_up),
    "bf16_bits truncates": (SG, "bf16_bits", m_bits_truncate),
    "bf16_bits ties to odd": (SG, "bf16_bits", m_bits_ties_odd),
}


@pytest.mark.parametrize("name", sorted(CODEC_MUTANTS))
def test_codec_mutant_is_caught(name, monkeypatch):
    mod, fn_name, fn = CODEC_MUTANTS[name]
    monkeypatch.setattr(mod, fn_name, fn)
    failed = _fails(ALL_CHECKS)
    assert failed, f"no pin catches the mutant {name!r}"
