"""Seeded synthetic sampling workloads (logits, per-row parameters, token histories, uniforms).

This package only draws random inputs.  It contains none of the sampling arithmetic, so both the CPU
oracle (``oracle/``) and the GPU path (``paper_2606_01927_amd``) can consume the same inputs without
sharing any code of the method itself.
"""
from .configs import (  # noqa: F401
    add_prompt,
    CONFIGS,
    Workload,
    generate,
    uniforms_from_u32,
    to_bf16_bits,
)
