"""Workload shapes for one DiT block on one GPU's share of a request.

The request classes follow the paper's evaluation workloads (section 6.1,
Experimental Setup): Wan2.2 videos of 480x832 and 720x1280 pixels with 81
frames, and Qwen-Image images of 1024x1024 and 1536x1536 pixels.  Token counts
assume 4x temporal and 8x spatial VAE compression followed by 1x2x2 patches
(2x2 for images); the paper states neither factor, so these counts are a
consistent reading, not a quotation:

* 480p video: latent 21x60x104 -> 21*30*52 = 32,760 tokens
* 720p video: latent 21x90x160 -> 21*45*80 = 75,600 tokens
* 1024^2 image: latent 128x128 -> 64*64 = 4,096 tokens
* 1536^2 image: latent 192x192 -> 96*96 = 9,216 tokens

Nothing here computes anything of the block; it is shared by the oracle and the
GPU path as plain data.
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int                         # seed component, fixed per workload
    dtype: str                       # "f32" or "bf16": storage and GEMM operand type
    hidden: int                      # D
    n_heads: int                     # H for the per-token stages (H*d == D)
    head_dim: int                    # d
    mlp_hidden: int                  # Dff
    freq_dim: int                    # F, width of the sinusoidal timestep encoding
    rope_sections: Tuple[int, int, int]   # (d_t, d_h, d_w); (0,0,0) disables rotary
    grids: Tuple[Tuple[int, int, int], ...]  # full (F, H, W) token grid per request
    rows: Tuple[int, ...]            # latent rows of each request on this GPU
    txt_len: int                     # text tokens per request
    attn_heads: Optional[int] = None     # heads of the self-attention stage if it differs (SP share)
    attn_rows: Optional[Tuple[int, ...]] = None  # full request lengths seen by self-attention (SP share)
    rope_theta: float = 10000.0
    ln_eps: float = 1e-6
    rms_eps: float = 1e-6
    linear_std: float = 0.02         # std of the Linear weight matrices
    description: str = ""

    @property
    def n_req(self) -> int:
        return len(self.rows)

    @property
    def n_rows(self) -> int:
        return sum(self.rows)

    @property
    def n_txt(self) -> int:
        return self.txt_len * self.n_req

    @property
    def is_sp_share(self) -> bool:
        return self.attn_rows is not None

    def cu_seqlens(self) -> List[int]:
        out = [0]
        for r in self.rows:
            out.append(out[-1] + r)
        return out

    def cu_txt(self) -> List[int]:
        return [i * self.txt_len for i in range(self.n_req + 1)]

    def cu_attn(self) -> List[int]:
        rows = self.attn_rows if self.attn_rows is not None else self.rows
        out = [0]
        for r in rows:
            out.append(out[-1] + r)
        return out


def _w(name, wid, dtype, D, H, d, Dff, F, sec, grids, rows, L, desc, **kw):
    return Workload(name=name, wid=wid, dtype=dtype, hidden=D, n_heads=H, head_dim=d,
                    mlp_hidden=Dff, freq_dim=F, rope_sections=sec, grids=tuple(grids),
                    rows=tuple(rows), txt_len=L, description=desc, **kw)


WORKLOADS: Dict[str, Workload] = {}
for _wl in [
    _w("tiny_image_fp32", 1, "f32", 384, 6, 64, 1536, 384, (0, 32, 32), [(1, 8, 8)], [64], 77,
       "tiny image block, fp32: 16x16x4 latent, patch 2 -> 64 tokens; D 384, 6x64 heads, "
       "MLP 1536, 77 text tokens"),
    _w("image_1024", 2, "bf16", 3072, 24, 128, 12288, 3072, (0, 64, 64), [(1, 64, 64)], [4096], 512,
       "1024x1024 image block, bf16: 128x128x16 latent, patch 2 -> 4,096 tokens; D 3072, "
       "24x128 heads, MLP 12288, 512 text tokens"),
    _w("video_480p", 3, "bf16", 5120, 40, 128, 13824, 5120, (44, 42, 42), [(21, 30, 52)], [32760], 512,
       "480p video block, bf16: latent 21x60x104x16, patch 1x2x2 -> 32,760 tokens; D 5120, "
       "40x128 heads, MLP 13824, 512 text tokens"),
    _w("video_720p", 4, "bf16", 5120, 40, 128, 13824, 5120, (44, 42, 42), [(21, 45, 80)], [75600], 512,
       "720p video block, bf16: latent 21x90x160x16, patch 1x2x2 -> 75,600 tokens; D 5120, "
       "40x128 heads, MLP 13824, 512 text tokens"),
    _w("packed_sp8_share", 5, "bf16", 5120, 40, 128, 13824, 5120, (44, 42, 42),
       [(1, 64, 64), (1, 96, 96), (21, 30, 52), (21, 45, 80)], [512, 1152, 4095, 9450], 512,
       "heterogeneous packed batch, one GPU's share at sequence-parallel degree 8: requests of "
       "4,096 / 9,216 / 32,760 / 75,600 tokens; per-token stages on the first 1/8 of each "
       "request's rows with all 40 heads; self-attention over the full lengths with 5 of 40 heads",
       attn_heads=5, attn_rows=(4096, 9216, 32760, 75600)),
]:
    WORKLOADS[_wl.name] = _wl


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from None


@dataclass(frozen=True)
class ModelWorkload:
    """One denoising step: a block workload (its requests must be whole) plus
    the model's depth, latent channels and patch size."""
    name: str
    block: Workload
    n_blocks: int
    in_channels: int
    patch: Tuple[int, int, int]
    description: str = ""

    @property
    def patch_len(self) -> int:
        return self.in_channels * self.patch[0] * self.patch[1] * self.patch[2]

    def latent_sizes(self) -> List[int]:
        pt, ph, pw = self.patch
        return [self.in_channels * f * pt * h * ph * w * pw for (f, h, w) in self.block.grids]


def _whole(name, wid, dtype, D, H, d, Dff, F, sec, grids, L, desc, **kw):
    rows = [f * h * w for (f, h, w) in grids]
    return _w(name, wid, dtype, D, H, d, Dff, F, sec, grids, rows, L, desc, **kw)


MODEL_WORKLOADS: Dict[str, ModelWorkload] = {}
for _mw in [
    ModelWorkload("step_tiny_fp32",
                  _whole("step_tiny_fp32.block", 11, "f32", 384, 6, 64, 1536, 384, (16, 24, 24),
                         [(2, 4, 6), (1, 8, 8)], 77, "two whole requests: 2x8x12 and 1x16x16 latents"),
                  2, 4, (1, 2, 2),
                  "tiny fp32 step: 2 blocks, 4 latent channels, patch 1x2x2, requests of 48 and 64 tokens"),
    ModelWorkload("step_small_bf16",
                  _whole("step_small_bf16.block", 12, "bf16", 256, 2, 128, 1024, 256, (44, 42, 42),
                         [(3, 4, 6), (1, 6, 10)], 40, "two whole requests: 3x8x12 and 1x12x20 latents; weight "
                         "matrices at std 0.02*sqrt(5120/256) so activations have the D = 5120 magnitudes",
                         linear_std=0.02 * (5120 / 256) ** 0.5),
                  2, 16, (1, 2, 2),
                  "small bf16 step: 2 blocks, D 256, 16 latent channels, patch 1x2x2, requests of 72 and 60 tokens"),
    ModelWorkload("step_image_1024", WORKLOADS["image_1024"], 60, 16, (1, 2, 2),
                  "1024x1024 image step: 60 blocks of the image block, latent 16x128x128, patch 1x2x2"),
    ModelWorkload("step_video_480p", WORKLOADS["video_480p"], 40, 16, (1, 2, 2),
                  "480p video step: 40 blocks of the 480p block, latent 16x21x60x104, patch 1x2x2"),
    ModelWorkload("step_video_720p", WORKLOADS["video_720p"], 40, 16, (1, 2, 2),
                  "720p video step: 40 blocks of the 720p block, latent 16x21x90x160, patch 1x2x2"),
]:
    MODEL_WORKLOADS[_mw.name] = _mw


def get_model_workload(name: str) -> ModelWorkload:
    try:
        return MODEL_WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown step workload {name!r}; known: {sorted(MODEL_WORKLOADS)}") from None


# Request classes of the paper's evaluation (section 6.1): Wan2.2 videos S/M/L
# (480x832 with 49 frames, 480x832 with 81 frames, 720x1280 with 81 frames) and
# Qwen-Image images S/M/L (512^2, 1024^2, 1536^2), with their SLO multipliers
# alpha.  Token counts use the same VAE/patch reading as the block workloads
# (49 frames -> 13 latent frames).  `model` names the block shape of the model
# that serves the class and `n_blocks` its depth.
@dataclass(frozen=True)
class RequestClass:
    name: str
    model: str          # "video" (D 5120, 40 x 128 heads) or "image" (D 3072, 24 x 128 heads)
    grid: Tuple[int, int, int]
    alpha: float
    n_steps: int = 50

    @property
    def tokens(self) -> int:
        return self.grid[0] * self.grid[1] * self.grid[2]


MODEL_SHAPES = {
    # hidden, heads, head_dim, mlp_hidden, freq_dim, rope sections, blocks, text tokens
    "video": (5120, 40, 128, 13824, 5120, (44, 42, 42), 40, 512),
    "image": (3072, 24, 128, 12288, 3072, (0, 64, 64), 60, 512),
}

REQUEST_CLASSES: Dict[str, RequestClass] = {c.name: c for c in [
    RequestClass("video_S", "video", (13, 30, 52), 2.0),
    RequestClass("video_M", "video", (21, 30, 52), 2.5),
    RequestClass("video_L", "video", (21, 45, 80), 3.5),
    RequestClass("image_S", "image", (1, 32, 32), 1.5),
    RequestClass("image_M", "image", (1, 64, 64), 2.0),
    RequestClass("image_L", "image", (1, 96, 96), 6.0),
]}
SP_DEGREES = (1, 2, 4, 8)


def share_workload(cls: RequestClass, degree: int) -> Workload:
    """One GPU's share of a class's block at sequence-parallel degree `degree`:
    per-token stages on the first ceil(n/degree) rows with all heads,
    self-attention over all n rows with heads/degree heads."""
    D, H, d, Dff, F, sec, _, L = MODEL_SHAPES[cls.model]
    n = cls.tokens
    rows = -(-n // degree)
    return Workload(name=f"{cls.name}.sp{degree}", wid=100 + degree, dtype="bf16", hidden=D, n_heads=H,
                    head_dim=d, mlp_hidden=Dff, freq_dim=F, rope_sections=sec, grids=(cls.grid,), rows=(rows,),
                    txt_len=L, attn_heads=H // degree if degree > 1 else None,
                    attn_rows=(n,) if degree > 1 else None,
                    description=f"{cls.name} at SP degree {degree}: {rows} of {n} rows, "
                                f"{H // degree} of {H} heads in self-attention")
