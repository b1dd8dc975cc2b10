"""CPU oracle (float64, NumPy) for one DiT block -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU path and
imports nothing from it; the only module both sides use is ``synth`` (seeded
inputs, no block arithmetic).  See ``oracle.dit_block`` for what is computed,
the readings it follows and how each part is pinned.
"""
from .dit_block import (
    BlockConfig, Varlen, decode, silu, gelu_tanh, linear, timestep_embedding,
    timestep_mlp, adaln_modulation, conditioning, layer_norm, modulate,
    rms_norm_heads, grid_positions, rope_angles, apply_rope, rope_for_rows,
    attention, attention_varlen, config_from_workload, varlen_from_workload,
    pre_attention, cross_kv, post_attention, block_forward, block_forward_rows,
)
