"""CPU oracle for the DiT denoising step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import anything from this package.  It shares no code with
the HIP library in ``paper_2510_01565_amd`` and imports nothing from it.
"""
from .dit_oracle import *  # noqa: F401,F403
from .dit_oracle import (OracleConfig, OracleRequest, attention, conditioning, dit_step,
                         dit_velocity, double_block, euler_update, final_layer, gelu_tanh,
                         image_tokens, layer_norm, linear, modulate, modulation,
                         modulation_layout, param_shapes, rope_2d, rope_angles, rotate_pairs,
                         silu, single_block, timestep_embedding)
