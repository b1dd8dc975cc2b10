"""CPU oracle for one denoising step of a DiT -- TEST INFRASTRUCTURE ONLY.

Like ``oracle.dit_block``, this is plain float64 NumPy that only the test
suite, ``__graft_entry__.smoke()`` and the CPU baseline leg of ``bench.py``
may import; the product path never calls it and shares no code with it.

What it computes.  The paper schedules DiT serving in trajectory tasks, one of
which is a single denoising step: it takes the latent state, the conditioning
and the text embeddings of a request and leaves the next latent state of its
diffusion trajectory (section 2.1, Rescheduling Boundaries; section 3.1,
Reschedulable Trajectory Tasks).  The paper does not define the model or the
sampler.  The step here is the standard DiT around the block of
``oracle.dit_block``, each part from its published definition:

* patch embedding and the adaLN final layer: Peebles & Xie, "Scalable
  Diffusion Models with Transformers" (DiT), 2023 -- non-overlapping
  pt x ph x pw patches flattened and projected by one Linear; the timestep MLP
  shared by all blocks; a final LayerNorm modulated by (shift, scale) =
  Linear(SiLU(c)) and a Linear back to patch values;
* the velocity field and its Euler step: rectified flow / flow matching
  (Liu et al., 2022; Lipman et al., 2022): on the path
  x_sigma = (1 - sigma) x_0 + sigma * noise the velocity is noise - x_0 and
  one Euler step from sigma to sigma' is x + (sigma' - sigma) * v.

Readings (R17..R22, continuing the block's R1..R16):
 R17 latent layout per request: channel-major [C, F*pt, H*ph, W*pw], the
     requests one after another;
 R18 token order (f, h, w) row-major, patch-vector order (c, i, j, k); the
     output projection uses the same order, so unpatchify inverts patchify;
 R19 one timestep MLP shared by all blocks; block b's modulation is
     W_ada_b SiLU(c) + b_ada_b (the DiT final layer takes the same SiLU(c));
 R20 final layer: LayerNorm without affine (eps ln_eps), modulated with
     (shift, scale) in that order, then Linear(D -> P);
 R21 the model's output is the velocity; the step is
     latent + dt * velocity with dt = sigma_next - sigma given per request;
 R22 the text keys and values of a block depend only on the text, so a cache
     of them (the GPU path's) equals recomputing them; the oracle recomputes.

Pins (tests/test_oracle_model.py): patchify against a brute-force loop and
against einops.rearrange; unpatchify(patchify(x)) == x exactly; the Euler
step lands exactly on the flow-matching path for the exact velocity; dt = 0
gives the latent back; zero output weights give the closed form
latent + dt * unpatchify(b_out); identity blocks (zero gates and zero cross
output) reduce the step to the embedding and head alone; the output is affine
in dt; with every block's own timestep MLP equal to the shared one, the
blocks inside the step equal oracle.dit_block.block_forward.
"""
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import dit_block as O


# ---------------------------------------------------------------------------
# latent <-> tokens (readings R17, R18)
# ---------------------------------------------------------------------------


def patchify(lat: np.ndarray, patch: Sequence[int]) -> np.ndarray:
    """One request's latent [C, F*pt, H*ph, W*pw] -> tokens [F*H*W, C*pt*ph*pw].
    Token (f, h, w) row-major; patch vector (c, i, j, k) row-major, where
    (i, j, k) is the offset inside the patch along (time, height, width)."""
    C, FL, HL, WL = lat.shape
    pt, ph, pw = patch
    F, H, W = FL // pt, HL // ph, WL // pw
    v = lat.reshape(C, F, pt, H, ph, W, pw)
    v = v.transpose(1, 3, 5, 0, 2, 4, 6)          # f, h, w, c, i, j, k
    return v.reshape(F * H * W, C * pt * ph * pw)


def unpatchify(tok: np.ndarray, C: int, grid: Tuple[int, int, int], patch: Sequence[int]) -> np.ndarray:
    """Inverse of ``patchify``: tokens [F*H*W, P] -> latent [C, F*pt, H*ph, W*pw]."""
    F, H, W = grid
    pt, ph, pw = patch
    v = tok.reshape(F, H, W, C, pt, ph, pw)
    v = v.transpose(3, 0, 4, 1, 5, 2, 6)          # c, f, i, h, j, w, k
    return v.reshape(C, F * pt, H * ph, W * pw)


def latent_sizes(C: int, grids: Sequence[Tuple[int, int, int]], patch: Sequence[int]) -> List[int]:
    """Values of each request's latent in the packed fp32 latent (R17)."""
    pt, ph, pw = patch
    return [C * f * pt * h * ph * w * pw for (f, h, w) in grids]


def split_latent(flat: np.ndarray, C: int, grids, patch) -> List[np.ndarray]:
    """Packed latent (1-D) -> per-request [C, F*pt, H*ph, W*pw] arrays."""
    out, off = [], 0
    pt, ph, pw = patch
    for (f, h, w), n in zip(grids, latent_sizes(C, grids, patch)):
        out.append(flat[off:off + n].reshape(C, f * pt, h * ph, w * pw))
        off += n
    return out


def patchify_packed(flat: np.ndarray, C: int, grids, patch) -> np.ndarray:
    """Packed latent -> packed tokens [sum F*H*W, P]."""
    return np.concatenate([patchify(l, patch) for l in split_latent(flat, C, grids, patch)], axis=0)


def unpatchify_packed(tok: np.ndarray, C: int, grids, patch) -> np.ndarray:
    """Packed tokens -> packed latent (1-D)."""
    out, row = [], 0
    for g in grids:
        n = g[0] * g[1] * g[2]
        out.append(unpatchify(tok[row:row + n], C, g, patch).reshape(-1))
        row += n
    return np.concatenate(out)


# ---------------------------------------------------------------------------
# conditioning, final layer, Euler step (readings R19..R21)
# ---------------------------------------------------------------------------


def shared_time(t: np.ndarray, freq_dim: int, mw: Dict[str, np.ndarray]) -> np.ndarray:
    """c = W_t2 SiLU(W_t1 emb(t) + b_t1) + b_t2 per request, the MLP shared by
    every block and the final layer (R19).  [R, D]."""
    e = O.timestep_embedding(t, freq_dim)
    return O.timestep_mlp(e, mw["w_t1"], mw["b_t1"], mw["w_t2"], mw["b_t2"])


def final_layer(x: np.ndarray, c: np.ndarray, req: np.ndarray, eps: float, mw: Dict[str, np.ndarray]) -> np.ndarray:
    """DiT final layer (R20): (shift, scale) = W_hmod SiLU(c) + b_hmod;
    v = (LN(x)(1 + scale) + shift) W_out^T + b_out.  [rows, P]."""
    m = O.linear(O.silu(c), mw["w_hmod"], mw["b_hmod"])
    D = x.shape[1]
    shift, scale = m[:, :D], m[:, D:]
    h = O.modulate(O.layer_norm(x, eps), shift[req], scale[req])
    return O.linear(h, mw["w_out"], mw["b_out"])


def euler_step(latent: np.ndarray, v: np.ndarray, dt) -> np.ndarray:
    """Flow-matching Euler update (R21): latent + dt * v."""
    return latent + dt * v


# ---------------------------------------------------------------------------
# the step
# ---------------------------------------------------------------------------


def denoise_step(cfg: O.BlockConfig, vl: O.Varlen, C: int, patch: Sequence[int], latent: np.ndarray,
                 t: np.ndarray, dt: np.ndarray, txt: np.ndarray, mw: Dict[str, np.ndarray],
                 blocks: Sequence[Dict[str, np.ndarray]], return_velocity: bool = False):
    """One Euler step of every request of a packed batch of whole requests.

    latent: packed fp32 values (R17), t and dt: [R], txt: [txt_rows, D],
    mw: the model's own weights (w_t1..b_t2, w_pe, b_pe, w_hmod, b_hmod,
    w_out, b_out), blocks: one weight dict per block (their w_t1..b_t2 are not
    used).  Returns the packed next latent (and the velocity tokens)."""
    grids = list(vl.grid_fhw)
    tok = patchify_packed(latent, C, grids, patch)
    x = O.linear(tok, mw["w_pe"], mw["b_pe"])
    c = shared_time(t, cfg.freq_dim, mw)
    for w in blocks:
        mod = O.adaln_modulation(c, w["w_ada"], w["b_ada"])
        x = O.block_forward(cfg, vl, x, t, txt, w, mod=mod)
    req = O._row_request(vl, x.shape[0])
    v = final_layer(x, c, req, cfg.ln_eps, mw)
    dt_el = np.concatenate([np.full(n, float(d)) for n, d in zip(latent_sizes(C, grids, patch), dt)])
    out = euler_step(latent, unpatchify_packed(v, C, grids, patch), dt_el)
    return (out, v) if return_velocity else out


def text_kv(cfg: O.BlockConfig, txt: np.ndarray, blocks: Sequence[Dict[str, np.ndarray]]) -> List[np.ndarray]:
    """Every block's cross-attention keys and values, [txt_rows, 2D] each (R22)."""
    out = []
    for w in blocks:
        ck, cv = O.cross_kv(cfg, txt, w)
        out.append(np.concatenate([ck, cv], axis=1))
    return out
