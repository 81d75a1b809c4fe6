"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This package holds no arithmetic of the method: it only defines workload
shapes and draws random numbers (weights, visual encodings, prompt ids,
schedules, batch shapes) from ``numpy.random.Generator(PCG64(seed))`` with
``seed = 1000 * config_id + stream`` (stream 0 weights, with ``+16 * layer``
per layer; 1 visual encoding; 2 prompt ids; 3 schedule; 4 batch shapes).
Rounding to bfloat16 (round-to-nearest-even) is part of input preparation:
the bf16 configurations hand both sides the same bf16-representable values.
"""

from .configs import CONFIGS, TEST_CONFIGS, Config, get_config, get_any_config  # noqa: F401,E501
from .gen import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    round_to_bf16,
    gen_visual,
    gen_prompt,
    gen_layer_weights,
    gen_embed,
    gen_head,
    gen_schedule,
    gen_batch_shapes,
    gen_sample,
)
