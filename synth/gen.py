"""Seeded generator for the block's inputs and weights.

Recipe (one fixed draw per named tensor, independent of generation order):

* every tensor has a stable id; its values are drawn with NumPy's PCG64 via
  ``default_rng([13501, workload_id, tensor_id, chunk])`` in chunks of
  ``CHUNK`` elements, so large tensors can be drawn on several threads and still
  give the same bits;
* standard normal draws in float32, scaled by the tensor's std and shifted by
  its mean, then stored either as float32 or as bfloat16 bits obtained by
  round-to-nearest-even on the float32 bit pattern;
* latents and text embeddings ~ N(0, 1); Linear weight matrices
  ~ N(0, linear_std^2) (0.02 for every workload shaped like the paper's);
  biases ~ N(0, 0.02^2); norm gains ~ 1 + N(0, 0.02^2); LayerNorm shift
  ~ N(0, 0.02^2); timesteps ~ U[0, 1000) (float32).

bfloat16 values travel as ``uint16`` arrays of their bit patterns.
"""
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Dict, Iterable, Optional, Sequence, Tuple
import os

import numpy as np

from .workloads import ModelWorkload, Workload

SEED = 13501
CHUNK = 1 << 22


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 bfloat16 bit patterns, round to nearest even."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


@dataclass(frozen=True)
class TensorSpec:
    name: str
    tid: int
    shape: Tuple[int, ...]
    dist: str           # "normal" or "uniform"
    mean: float = 0.0
    std: float = 1.0
    lo: float = 0.0
    hi: float = 1.0
    dtype: Optional[str] = None   # None: the workload's dtype; "f32" forces float32


def _fill(spec: TensorSpec, wid: int, threads: int, as_bf16: bool) -> np.ndarray:
    n = int(np.prod(spec.shape)) if spec.shape else 1
    out = np.empty(n, dtype=np.uint16 if as_bf16 else np.float32)
    chunks = [(c, c * CHUNK, min(n, (c + 1) * CHUNK)) for c in range((n + CHUNK - 1) // CHUNK)]

    def work(ch):
        c, a, b = ch
        rng = np.random.default_rng([SEED, wid, spec.tid, c])
        if spec.dist == "normal":
            v = rng.standard_normal(b - a, dtype=np.float32)
            if spec.std != 1.0:
                v *= np.float32(spec.std)
            if spec.mean != 0.0:
                v += np.float32(spec.mean)
        elif spec.dist == "uniform":
            v = rng.random(b - a, dtype=np.float32)
            v = (v * np.float32(spec.hi - spec.lo) + np.float32(spec.lo)).astype(np.float32)
            # guard the half-open interval against rounding up to hi
            v = np.minimum(v, np.nextafter(np.float32(spec.hi), np.float32(spec.lo)))
        else:
            raise ValueError(spec.dist)
        out[a:b] = bf16_bits(v) if as_bf16 else v

    if len(chunks) > 1 and threads > 1:
        with ThreadPoolExecutor(min(threads, len(chunks))) as ex:
            list(ex.map(work, chunks))
    else:
        for ch in chunks:
            work(ch)
    return out.reshape(spec.shape)


def generate_tensor(spec: TensorSpec, wl: Workload, threads: Optional[int] = None) -> np.ndarray:
    threads = threads or min(16, os.cpu_count() or 1)
    dt = spec.dtype or wl.dtype
    if dt not in ("f32", "bf16"):
        raise ValueError(dt)
    return _fill(spec, wl.wid, threads, dt == "bf16")


def block_tensor_specs(wl: Workload) -> Dict[str, TensorSpec]:
    """All inputs and weights of one block, keyed by name ([out, in] weights)."""
    D, F, Dff, d = wl.hidden, wl.freq_dim, wl.mlp_hidden, wl.head_dim
    W = wl.linear_std
    specs = [
        TensorSpec("x", 1, (wl.n_rows, D), "normal"),
        TensorSpec("txt", 2, (wl.n_txt, D), "normal"),
        TensorSpec("t", 3, (wl.n_req,), "uniform", lo=0.0, hi=1000.0, dtype="f32"),
        TensorSpec("w_t1", 10, (D, F), "normal", std=W),
        TensorSpec("b_t1", 11, (D,), "normal", std=0.02),
        TensorSpec("w_t2", 12, (D, D), "normal", std=W),
        TensorSpec("b_t2", 13, (D,), "normal", std=0.02),
        TensorSpec("w_ada", 14, (6 * D, D), "normal", std=W),
        TensorSpec("b_ada", 15, (6 * D,), "normal", std=0.02),
        TensorSpec("w_qkv", 16, (3 * D, D), "normal", std=W),
        TensorSpec("b_qkv", 17, (3 * D,), "normal", std=0.02),
        TensorSpec("g_q", 18, (d,), "normal", mean=1.0, std=0.02),
        TensorSpec("g_k", 19, (d,), "normal", mean=1.0, std=0.02),
        TensorSpec("w_o", 20, (D, D), "normal", std=W),
        TensorSpec("b_o", 21, (D,), "normal", std=0.02),
        TensorSpec("g_ca", 22, (D,), "normal", mean=1.0, std=0.02),
        TensorSpec("b_ca", 23, (D,), "normal", std=0.02),
        TensorSpec("w_cq", 24, (D, D), "normal", std=W),
        TensorSpec("b_cq", 25, (D,), "normal", std=0.02),
        TensorSpec("w_ckv", 26, (2 * D, D), "normal", std=W),
        TensorSpec("b_ckv", 27, (2 * D,), "normal", std=0.02),
        TensorSpec("g_cq", 28, (d,), "normal", mean=1.0, std=0.02),
        TensorSpec("g_ck", 29, (d,), "normal", mean=1.0, std=0.02),
        TensorSpec("w_co", 30, (D, D), "normal", std=W),
        TensorSpec("b_co", 31, (D,), "normal", std=0.02),
        TensorSpec("w_up", 32, (Dff, D), "normal", std=W),
        TensorSpec("b_up", 33, (Dff,), "normal", std=0.02),
        TensorSpec("w_dn", 34, (D, Dff), "normal", std=W),
        TensorSpec("b_dn", 35, (D,), "normal", std=0.02),
    ]
    return {s.name: s for s in specs}


WEIGHT_NAMES = (
    "w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada", "w_qkv", "b_qkv", "g_q", "g_k",
    "w_o", "b_o", "g_ca", "b_ca", "w_cq", "b_cq", "w_ckv", "b_ckv", "g_cq", "g_ck",
    "w_co", "b_co", "w_up", "b_up", "w_dn", "b_dn",
)


def generate_block_inputs(wl: Workload, names: Optional[Iterable[str]] = None,
                          threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    specs = block_tensor_specs(wl)
    names = list(names) if names is not None else list(specs)
    return {n: generate_tensor(specs[n], wl, threads) for n in names}


def generate_attention_inputs(wl: Workload, threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Synthetic q, k, v ~ N(0, 1) for the self-attention stage on its own.

    Shapes are [rows, heads, head_dim] over the lengths and heads the attention
    stage sees (the full request lengths and the head share for an SP share).
    Also an attention output ``o`` ~ N(0, 1) of shape [rows, D] for the
    post-attention stage of an SP share, whose producer (the exchange of heads
    for rows between GPUs) is not part of one GPU's work.
    """
    heads = wl.attn_heads or wl.n_heads
    n_attn = wl.cu_attn()[-1]
    specs = {
        "q": TensorSpec("q", 40, (n_attn, heads, wl.head_dim), "normal"),
        "k": TensorSpec("k", 41, (n_attn, heads, wl.head_dim), "normal"),
        "v": TensorSpec("v", 42, (n_attn, heads, wl.head_dim), "normal"),
        "o": TensorSpec("o", 43, (wl.n_rows, wl.hidden), "normal"),
    }
    return {n: generate_tensor(s, wl, threads) for n, s in specs.items()}


def generate_sampled_rows(wl: Workload, n_per_req: int, sample_id: int = 0,
                          attn: bool = False, tile: Optional[int] = None) -> np.ndarray:
    """Sorted global row indices: a seeded sample of each request's rows that
    always includes the first and last row and rows at frame boundaries, and
    with ``tile`` also the first and last row of every ``tile``-row block of
    the packed batch (global row index) that the request touches."""
    rng = np.random.default_rng([SEED, wl.wid, 1000 + sample_id])
    cu = wl.cu_attn() if attn else wl.cu_seqlens()
    out = []
    for r in range(wl.n_req):
        n = cu[r + 1] - cu[r]
        Fg, Hg, Wg = wl.grids[r]
        must = {0, n - 1}
        frame = Hg * Wg
        for f in range(1, Fg):
            if f * frame < n:
                must.add(f * frame - 1)
                must.add(f * frame)
        if tile:
            for g in range(cu[r] // tile * tile, cu[r + 1], tile):
                for row in (g, g + tile - 1):
                    if cu[r] <= row < cu[r + 1]:
                        must.add(row - cu[r])
        must = sorted(must)[: max(2, n_per_req // 2)]
        k = max(0, min(n, n_per_req) - len(must))
        pool = np.setdiff1d(np.arange(n), np.array(must))
        pick = rng.choice(pool, size=min(k, len(pool)), replace=False) if k else np.array([], int)
        rows = np.unique(np.concatenate([np.array(must, dtype=np.int64), pick.astype(np.int64)]))
        out.append(rows + cu[r])
    return np.concatenate(out)


def draw(shape, key: Sequence[int], dtype: str = "bf16", dist: str = "normal", mean: float = 0.0,
         std: float = 1.0, lo: float = 0.0, hi: float = 1.0, threads: Optional[int] = None) -> np.ndarray:
    """A free-standing seeded tensor (same recipe, seed [13501, 900, *key, chunk])."""
    class _W:
        wid = 900
    spec = TensorSpec("draw", 0, tuple(int(s) for s in shape), dist, mean=mean, std=std, lo=lo, hi=hi)
    threads = threads or min(16, os.cpu_count() or 1)
    n = int(np.prod(spec.shape)) if spec.shape else 1
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    chunks = [(c, c * CHUNK, min(n, (c + 1) * CHUNK)) for c in range((n + CHUNK - 1) // CHUNK)]

    def work(ch):
        c, a, b = ch
        rng = np.random.default_rng([SEED, 900] + [int(k) for k in key] + [c])
        if dist == "normal":
            v = rng.standard_normal(b - a, dtype=np.float32) * np.float32(std) + np.float32(mean)
        else:
            v = (rng.random(b - a, dtype=np.float32) * np.float32(hi - lo) + np.float32(lo)).astype(np.float32)
        out[a:b] = bf16_bits(v) if dtype == "bf16" else v

    if len(chunks) > 1 and threads > 1:
        with ThreadPoolExecutor(min(threads, len(chunks))) as ex:
            list(ex.map(work, chunks))
    else:
        for ch in chunks:
            work(ch)
    return out.reshape(spec.shape)


MODEL_WEIGHT_NAMES = ("w_t1", "b_t1", "w_t2", "b_t2", "w_pe", "b_pe", "w_hmod", "b_hmod", "w_out", "b_out")


def model_tensor_specs(mw: ModelWorkload) -> Dict[str, TensorSpec]:
    """The step's own inputs and weights: the packed fp32 latent ~ N(0, 1),
    t ~ U[0, 1000), dt ~ U[-0.05, -0.01) (one step of a 20..100-step schedule
    towards sigma = 0), and the model-level weights."""
    wl = mw.block
    D, F, P = wl.hidden, wl.freq_dim, mw.patch_len
    W = wl.linear_std
    specs = [
        TensorSpec("latent", 50, (sum(mw.latent_sizes()),), "normal", dtype="f32"),
        TensorSpec("t", 51, (wl.n_req,), "uniform", lo=0.0, hi=1000.0, dtype="f32"),
        TensorSpec("dt", 52, (wl.n_req,), "uniform", lo=-0.05, hi=-0.01, dtype="f32"),
        TensorSpec("txt", 2, (wl.n_txt, D), "normal"),
        TensorSpec("w_t1", 53, (D, F), "normal", std=W),
        TensorSpec("b_t1", 54, (D,), "normal", std=0.02),
        TensorSpec("w_t2", 55, (D, D), "normal", std=W),
        TensorSpec("b_t2", 56, (D,), "normal", std=0.02),
        TensorSpec("w_pe", 57, (D, P), "normal", std=W),
        TensorSpec("b_pe", 58, (D,), "normal", std=0.02),
        TensorSpec("w_hmod", 59, (2 * D, D), "normal", std=W),
        TensorSpec("b_hmod", 60, (2 * D,), "normal", std=0.02),
        TensorSpec("w_out", 61, (P, D), "normal", std=W),
        TensorSpec("b_out", 62, (P,), "normal", std=0.02),
    ]
    return {s.name: s for s in specs}


def generate_model_inputs(mw: ModelWorkload, threads: Optional[int] = None, n_blocks: Optional[int] = None):
    """(model tensors, [block weight dicts]).  Block b's weights use the block
    recipe with tensor ids offset by 1000 * (b + 1); they omit the blocks' own
    timestep MLP, which the step does not read.  n_blocks: only the first
    n_blocks blocks (their values do not depend on how many are drawn)."""
    specs = model_tensor_specs(mw)
    model = {n: generate_tensor(s, mw.block, threads) for n, s in specs.items()}
    bspecs = block_tensor_specs(mw.block)
    blocks = []
    for b in range(mw.n_blocks if n_blocks is None else n_blocks):
        d = {}
        for n in WEIGHT_NAMES:
            if n in ("w_t1", "b_t1", "w_t2", "b_t2"):
                continue
            s = bspecs[n]
            d[n] = generate_tensor(TensorSpec(s.name, s.tid + 1000 * (b + 1), s.shape, s.dist, s.mean, s.std,
                                              s.lo, s.hi, s.dtype), mw.block, threads)
        blocks.append(d)
    return model, blocks
