"""CPU oracle for one DiT transformer block -- TEST INFRASTRUCTURE ONLY.

This module is the plain, slow, float64 reference that every GPU result is
checked against.  Only the test suite, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import it; the product path (the C-ABI
library and its Python binding) never calls it and shares no code with it.

What it computes.  The paper (GF-DiT, "Scheduling Parallelism for Diffusion
Transformer Serving") states that the denoising stage dominates execution
time (section 1, Introduction) and that a denoising step performs
bidirectional computation over the entire latent sequence (section 2.1,
Rescheduling Boundaries); its evaluation serves Wan2.2-5B and Qwen-Image
(section 6.1, Experimental Setup).  It does not define the block's internals.
The block here is the adaLN-Zero DiT block with QK-RMSNorm, sectioned 3D
rotary embeddings, full non-causal self-attention, cross-attention to text and
a GELU-tanh MLP, each written from its standard published definition:

* adaLN-Zero modulation and the sinusoidal timestep embedding: Peebles & Xie,
  "Scalable Diffusion Models with Transformers" (DiT), 2023;
* LayerNorm: Ba, Kiros & Hinton, 2016 (biased variance, epsilon inside the root);
* RMSNorm: Zhang & Sennrich, 2019;
* rotary position embedding: Su et al., RoFormer, 2021 (adjacent-pair rotation),
  split into (t, h, w) sections of the head dimension;
* scaled dot-product attention: Vaswani et al., 2017;
* GELU with the tanh approximation: Hendrycks & Gimpel, 2016.

Where the paper is silent the numbered readings R1..R16 apply; each function
names the ones it follows.  Everything runs in float64 from the stored input
values; no intermediate is rounded.  Contractions use ``numpy.matmul``.

Pins (tests/test_oracle_*.py): brute-force loops on tiny inputs, closed forms
of special cases, invariants (softmax rows sum to one, rotary preserves norms
and depends on relative position only, zero gates give an identity block,
permutation equivariance without rotary) and library cross-checks
(torch float64 layer_norm, rms_norm, scaled_dot_product_attention, gelu).
The composition of the whole block (which stage follows which) has no printed
example in the paper: parity unpinned by the paper; it is pinned only by the
readings plus the closed-form wiring tests and invariants.
"""
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# input decoding (storage formats -> float64)
# ---------------------------------------------------------------------------


def decode(a: np.ndarray) -> np.ndarray:
    """Stored value -> float64.  uint16 arrays hold bfloat16 bit patterns."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


@dataclass
class BlockConfig:
    """Hyper-parameters of one block (mirrors the fields of the C header)."""
    hidden: int
    n_heads: int
    head_dim: int
    mlp_hidden: int
    freq_dim: int
    rope_sections: Tuple[int, int, int]
    rope_theta: float = 10000.0
    ln_eps: float = 1e-6
    rms_eps: float = 1e-6
    qk_norm: bool = True


@dataclass
class Varlen:
    """Packed batch: request r owns rows cu_seqlens[r]..cu_seqlens[r+1] and
    text rows cu_txt[r]..cu_txt[r+1]; grid_fhw[r] is its full (F, H, W) token
    grid and pos_offset[r] the flattened grid index of its first row here."""
    cu_seqlens: Sequence[int]
    cu_txt: Sequence[int]
    grid_fhw: Sequence[Tuple[int, int, int]]
    pos_offset: Optional[Sequence[int]] = None

    @property
    def n_req(self) -> int:
        return len(self.cu_seqlens) - 1

    def offset(self, r: int) -> int:
        return 0 if self.pos_offset is None else int(self.pos_offset[r])


# ---------------------------------------------------------------------------
# elementwise pieces
# ---------------------------------------------------------------------------


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z)."""
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation (Hendrycks & Gimpel):
    0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def linear(z: np.ndarray, w: np.ndarray, b: Optional[np.ndarray]) -> np.ndarray:
    """z W^T + b with W stored [out, in] (PyTorch Linear layout)."""
    y = np.matmul(z, w.T)
    if b is not None:
        y = y + b
    return y


# ---------------------------------------------------------------------------
# S0: timestep conditioning -> six modulation vectors (readings R2, R9)
# ---------------------------------------------------------------------------


def timestep_embedding(t: np.ndarray, freq_dim: int, max_period: float = 10000.0) -> np.ndarray:
    """Sinusoidal encoding of a scalar timestep (DiT): half = F/2 frequencies
    w_i = max_period^(-i/half), output [cos(t w), sin(t w)] (reading R9)."""
    t = np.asarray(t, dtype=np.float64).reshape(-1)
    half = freq_dim // 2
    i = np.arange(half, dtype=np.float64)
    w = np.exp(-np.log(max_period) * i / half)
    arg = t[:, None] * w[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=1)


def timestep_mlp(e: np.ndarray, w_t1, b_t1, w_t2, b_t2) -> np.ndarray:
    """c = W2 SiLU(W1 e + b1) + b2 (reading R9)."""
    return linear(silu(linear(e, w_t1, b_t1)), w_t2, b_t2)


def adaln_modulation(c: np.ndarray, w_ada, b_ada) -> np.ndarray:
    """adaLN-Zero: m = W_ada SiLU(c) + b_ada, split into six D-vectors in the
    order shift_sa, scale_sa, gate_sa, shift_ff, scale_ff, gate_ff (reading R2).
    Returns [R, 6, D]."""
    m = linear(silu(c), w_ada, b_ada)
    return m.reshape(m.shape[0], 6, -1)


def conditioning(t: np.ndarray, freq_dim: int, w: Dict[str, np.ndarray]) -> np.ndarray:
    """S0: per-request timestep -> modulation [R, 6, D]."""
    e = timestep_embedding(t, freq_dim)
    c = timestep_mlp(e, w["w_t1"], w["b_t1"], w["w_t2"], w["b_t2"])
    return adaln_modulation(c, w["w_ada"], w["b_ada"])


# ---------------------------------------------------------------------------
# normalisations (readings R4, R5, R6)
# ---------------------------------------------------------------------------


def layer_norm(z: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis without affine: (z - mean) / sqrt(var + eps),
    biased variance (reading R5)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return (z - mu) / np.sqrt(var + eps)


def modulate(hn: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """adaLN: hn * (1 + scale) + shift (reading R2)."""
    return hn * (1.0 + scale) + shift


def rms_norm_heads(u: np.ndarray, gamma: np.ndarray, n_heads: int, head_dim: int,
                   eps: float) -> np.ndarray:
    """RMSNorm applied to each head's head_dim values separately with a gain
    gamma of length head_dim (reading R6): u / sqrt(mean(u^2) + eps) * gamma."""
    n = u.shape[0]
    v = u.reshape(n, n_heads, head_dim)
    ms = (v * v).mean(axis=-1, keepdims=True)
    return (v / np.sqrt(ms + eps) * gamma).reshape(n, n_heads * head_dim)


# ---------------------------------------------------------------------------
# rotary position embedding over (t, h, w) sections (reading R7)
# ---------------------------------------------------------------------------


def grid_positions(n_rows: int, grid_fhw: Tuple[int, int, int], offset: int = 0) -> np.ndarray:
    """Integer (p_t, p_h, p_w) of rows 0..n-1 of a request whose first row has
    flattened grid index ``offset`` (row-major over F, H, W).  [n, 3]."""
    _, Hg, Wg = grid_fhw
    g = np.arange(n_rows, dtype=np.int64) + int(offset)
    return np.stack([g // (Hg * Wg), (g // Wg) % Hg, g % Wg], axis=1)


def rope_angles(pos: np.ndarray, sections: Tuple[int, int, int], theta: float) -> np.ndarray:
    """Angle of every adjacent pair of the head dim: pair j of section s has
    angle p_s * theta^(-2j/d_s).  Returns [n, head_dim/2] (reading R7)."""
    cols = []
    for s, ds in enumerate(sections):
        if ds == 0:
            continue
        j = np.arange(ds // 2, dtype=np.float64)
        inv = theta ** (-2.0 * j / ds)
        cols.append(pos[:, s:s + 1].astype(np.float64) * inv[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(u: np.ndarray, n_heads: int, head_dim: int, angles: np.ndarray) -> np.ndarray:
    """Rotate each adjacent pair (u[2i], u[2i+1]) of every head by its angle:
    (a, b) -> (a cos - b sin, a sin + b cos) (reading R7)."""
    n = u.shape[0]
    v = u.reshape(n, n_heads, head_dim // 2, 2)
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    a, b = v[..., 0], v[..., 1]
    out = np.stack([a * c - b * s, a * s + b * c], axis=-1)
    return out.reshape(n, n_heads * head_dim)


def rope_for_rows(u: np.ndarray, cfg: BlockConfig, vl: Varlen) -> np.ndarray:
    """Apply the sectioned rotary embedding to packed rows (all requests)."""
    if sum(cfg.rope_sections) == 0:
        return u
    out = np.empty_like(u)
    for r in range(vl.n_req):
        a, b = vl.cu_seqlens[r], vl.cu_seqlens[r + 1]
        pos = grid_positions(b - a, vl.grid_fhw[r], vl.offset(r))
        ang = rope_angles(pos, cfg.rope_sections, cfg.rope_theta)
        out[a:b] = apply_rope(u[a:b], cfg.n_heads, cfg.head_dim, ang)
    return out


# ---------------------------------------------------------------------------
# attention (reading R10)
# ---------------------------------------------------------------------------


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
              q_chunk: int = 1024) -> np.ndarray:
    """softmax(q k^T * scale) v for one head, no mask, non-causal.  The score
    matrix is materialised per chunk of query rows; softmax subtracts the row
    maximum and normalises exactly."""
    out = np.empty((q.shape[0], v.shape[1]), dtype=np.float64)
    for a in range(0, q.shape[0], q_chunk):
        s = np.matmul(q[a:a + q_chunk], k.T) * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[a:a + q_chunk] = np.matmul(p, v)
    return out


def attention_varlen(q: np.ndarray, k: np.ndarray, v: np.ndarray, cu_q: Sequence[int],
                     cu_k: Sequence[int], n_heads: int, head_dim: int,
                     scale: Optional[float] = None, q_rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Packed multi-head attention: request r's queries (rows cu_q[r]..) attend
    only to its keys (rows cu_k[r]..).  q, k, v are [rows, H*d] (head j in
    columns j*d..(j+1)*d).  With ``q_rows`` (sorted global query rows) only
    those output rows are computed, still over all of each request's keys."""
    scale = 1.0 / np.sqrt(head_dim) if scale is None else scale
    nq = q.shape[0] if q_rows is None else len(q_rows)
    out = np.zeros((nq, n_heads * head_dim), dtype=np.float64)
    for r in range(len(cu_q) - 1):
        qa, qb, ka, kb = cu_q[r], cu_q[r + 1], cu_k[r], cu_k[r + 1]
        if q_rows is None:
            sel_out = np.arange(qa, qb)
            sel_q = sel_out
        else:
            m = (q_rows >= qa) & (q_rows < qb)
            sel_out = np.nonzero(m)[0]
            sel_q = q_rows[m]
        if len(sel_q) == 0:
            continue
        for h in range(n_heads):
            cs = slice(h * head_dim, (h + 1) * head_dim)
            out[sel_out, cs] = attention(q[sel_q, cs], k[ka:kb, cs], v[ka:kb, cs], scale)
    return out


# ---------------------------------------------------------------------------
# the block (readings R1..R12)
# ---------------------------------------------------------------------------


def config_from_workload(wl) -> BlockConfig:
    return BlockConfig(hidden=wl.hidden, n_heads=wl.n_heads, head_dim=wl.head_dim,
                       mlp_hidden=wl.mlp_hidden, freq_dim=wl.freq_dim,
                       rope_sections=tuple(wl.rope_sections), rope_theta=wl.rope_theta,
                       ln_eps=wl.ln_eps, rms_eps=wl.rms_eps)


def varlen_from_workload(wl) -> Varlen:
    return Varlen(cu_seqlens=wl.cu_seqlens(), cu_txt=wl.cu_txt(), grid_fhw=list(wl.grids))


def _row_request(vl: Varlen, n_rows: int) -> np.ndarray:
    req = np.empty(n_rows, dtype=np.int64)
    for r in range(vl.n_req):
        req[vl.cu_seqlens[r]:vl.cu_seqlens[r + 1]] = r
    return req


def pre_attention(cfg: BlockConfig, vl: Varlen, x: np.ndarray, w: Dict[str, np.ndarray],
                  mod: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Steps before self-attention: modulated LayerNorm, QKV projection,
    per-head RMSNorm of q and k, rotary on q and k.  Returns q, k, v [rows, D]."""
    D = cfg.hidden
    req = _row_request(vl, x.shape[0])
    h = modulate(layer_norm(x, cfg.ln_eps), mod[req, 0], mod[req, 1])
    qkv = linear(h, w["w_qkv"], w["b_qkv"])
    q, k, v = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]
    if cfg.qk_norm:
        q = rms_norm_heads(q, w["g_q"], cfg.n_heads, cfg.head_dim, cfg.rms_eps)
        k = rms_norm_heads(k, w["g_k"], cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    q = rope_for_rows(q, cfg, vl)
    k = rope_for_rows(k, cfg, vl)
    return q, k, v


def cross_kv(cfg: BlockConfig, txt: np.ndarray, w: Dict[str, np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """Text keys and values of the cross-attention (reading R10): [cK|cV] =
    C W_ckv^T + b_ckv, RMSNorm on cK per head, no rotary."""
    D = cfg.hidden
    ckv = linear(txt, w["w_ckv"], w["b_ckv"])
    ck, cv = ckv[:, :D], ckv[:, D:]
    if cfg.qk_norm:
        ck = rms_norm_heads(ck, w["g_ck"], cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    return ck, cv


def post_attention(cfg: BlockConfig, vl: Varlen, x: np.ndarray, o: np.ndarray, txt: np.ndarray,
                   w: Dict[str, np.ndarray], mod: np.ndarray) -> np.ndarray:
    """Steps after self-attention, all per row given the attention output o:
    gated output projection, cross-attention to the request's text, gated MLP.
    Readings R1 (order), R3 (ungated cross residual), R4 (affine LayerNorm
    before cross-attention), R6 (RMSNorm on cq and ck), R11..R12."""
    D = cfg.hidden
    req = _row_request(vl, x.shape[0])
    x1 = x + mod[req, 2] * linear(o, w["w_o"], w["b_o"])
    hc = layer_norm(x1, cfg.ln_eps) * w["g_ca"] + w["b_ca"]
    cq = linear(hc, w["w_cq"], w["b_cq"])
    if cfg.qk_norm:
        cq = rms_norm_heads(cq, w["g_cq"], cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    ck, cv = cross_kv(cfg, txt, w)
    oc = attention_varlen(cq, ck, cv, vl.cu_seqlens, vl.cu_txt, cfg.n_heads, cfg.head_dim)
    x2 = x1 + linear(oc, w["w_co"], w["b_co"])
    h2 = modulate(layer_norm(x2, cfg.ln_eps), mod[req, 3], mod[req, 4])
    u = gelu_tanh(linear(h2, w["w_up"], w["b_up"]))
    return x2 + mod[req, 5] * linear(u, w["w_dn"], w["b_dn"])


def block_forward(cfg: BlockConfig, vl: Varlen, x: np.ndarray, t: np.ndarray, txt: np.ndarray,
                  w: Dict[str, np.ndarray], mod: Optional[np.ndarray] = None) -> np.ndarray:
    """One DiT block over a packed batch (reading R1): conditioning, modulated
    LayerNorm, QKV, QK-RMSNorm, rotary, self-attention within each request,
    gated output projection, cross-attention, gated GELU-tanh MLP."""
    if mod is None:
        mod = conditioning(t, cfg.freq_dim, w)
    q, k, v = pre_attention(cfg, vl, x, w, mod)
    o = attention_varlen(q, k, v, vl.cu_seqlens, vl.cu_seqlens, cfg.n_heads, cfg.head_dim)
    return post_attention(cfg, vl, x, o, txt, w, mod)


def block_forward_rows(cfg: BlockConfig, vl: Varlen, x: np.ndarray, t: np.ndarray,
                       txt: np.ndarray, w: Dict[str, np.ndarray], rows: np.ndarray,
                       mod: Optional[np.ndarray] = None, row_chunk: int = 8192) -> np.ndarray:
    """The block's output for the sorted global rows ``rows`` only.  Keys and
    values need every row, so the pre-attention steps run on all rows (in
    chunks of ``row_chunk``); attention and the per-row steps after it run on
    the requested rows.  Equal to ``block_forward(...)[rows]``."""
    if mod is None:
        mod = conditioning(t, cfg.freq_dim, w)
    n, D = x.shape
    k_all = np.empty((n, D))
    v_all = np.empty((n, D))
    q_sel = np.empty((len(rows), D))
    req = _row_request(vl, n)
    for a in range(0, n, row_chunk):
        b = min(n, a + row_chunk)
        # the chunk as its own packed batch: same requests, clipped rows, shifted offsets
        sub_cu, sub_off, sub_grid, sub_req = [0], [], [], []
        for r in range(vl.n_req):
            lo, hi = max(a, vl.cu_seqlens[r]), min(b, vl.cu_seqlens[r + 1])
            if lo < hi:
                sub_cu.append(sub_cu[-1] + hi - lo)
                sub_off.append(vl.offset(r) + lo - vl.cu_seqlens[r])
                sub_grid.append(vl.grid_fhw[r])
                sub_req.append(r)
        sub = Varlen(sub_cu, [0] * len(sub_cu), sub_grid, sub_off)
        q, k, v = pre_attention(cfg, sub, x[a:b], w, mod[sub_req])
        k_all[a:b], v_all[a:b] = k, v
        m = (rows >= a) & (rows < b)
        q_sel[np.nonzero(m)[0]] = q[rows[m] - a]
    o_sel = np.zeros((len(rows), D))
    for r in range(vl.n_req):
        qa, qb, ka, kb = vl.cu_seqlens[r], vl.cu_seqlens[r + 1], vl.cu_seqlens[r], vl.cu_seqlens[r + 1]
        m = np.nonzero((rows >= qa) & (rows < qb))[0]
        if len(m) == 0:
            continue
        for h in range(cfg.n_heads):
            cs = slice(h * cfg.head_dim, (h + 1) * cfg.head_dim)
            o_sel[m, cs] = attention(q_sel[m, cs], k_all[ka:kb, cs], v_all[ka:kb, cs],
                                     1.0 / np.sqrt(cfg.head_dim))
    # post-attention steps are per row: run them on the selected rows as a packed batch
    sel_cu, sel_req = [0], []
    for r in range(vl.n_req):
        cnt = int(((rows >= vl.cu_seqlens[r]) & (rows < vl.cu_seqlens[r + 1])).sum())
        sel_cu.append(sel_cu[-1] + cnt)
        sel_req.append(r)
    sel = Varlen(sel_cu, vl.cu_txt, vl.grid_fhw)
    return post_attention(cfg, sel, x[rows], o_sel, txt, w, mod)
