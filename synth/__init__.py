"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds shapes, seeds and random draws only; none of the method's arithmetic.
"""
from .configs import (Workload, TINY, SMALL, WAN14B_480P, WAN14B_720P, ALL,
                      SWEEP_RATIOS, SWEEP_AUDIO, sweep)
from .inputs import (make_audio, make_latents, make_block_weights, random_frame_weight,
                     random_anchor_keys, make_wan_block_weights, make_context,
                     to_bf16_bits, bf16_bits_to_f32, storage_round)
