"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

Holds no arithmetic of the method itself; see ``synth.gen``.
"""
from .gen import (Workload, tiny, llama8b_1layer, llama8b_32layer, ragged,  # noqa: F401
                  kv_rows, q_row, logits_row, hh_axes, hh_mask, hh_relevance_bounds,
                  bf16_bits, bf16_to_f32, round_to)
