"""Seeded synthetic workloads for the rolling denoise step.

This module only *draws* inputs: model shapes, weights, prefix key/value
contexts, observation vectors and stand-in FOP tokens. It holds none of the
method's arithmetic; the CPU oracle and the GPU library both consume what it
returns, and neither imports the other.

Every array is drawn from numpy's PCG64 generator seeded by
``SeedSequence(seed, spawn_key=(crc32(tag), ...))`` so that any tensor can be
regenerated on its own, in any order, on any machine.
"""

from .workloads import (  # noqa: F401
    CONFIGS,
    RavelShape,
    bf16_round,
    context_schedule,
    draw_context,
    draw_fop_tokens,
    draw_observation,
    draw_weights,
    get_config,
    param_count,
    weight_shapes,
)
