"""MI355X (gfx950) DiT block forward: hand-written HIP kernels behind a C ABI.

``binding`` holds the ctypes wrappers of ``include/dit_block.h``.  The HIP
library ``libditblock.so`` must have been built (``build.build()``); without
it every entry point raises ``binding.ExtensionMissing``.
"""
from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    BlockConfig, Varlen, DitError, ExtensionMissing, make_weights, block_workspace_size,
    block_forward, block_pre_attention, block_post_attention, timestep_modulation, timestep_modulation_noalloc,
    attention_varlen, adaln_modulate, layer_norm_affine, linear, qk_norm_rope, gated_residual,
)
