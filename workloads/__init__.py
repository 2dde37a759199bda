"""Seeded synthetic inputs for the integer relative-position attention block.

This package is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It draws the integer tensors, the real-valued quantization scales and
the sequence lengths, and turns the scales into the fixed-point integers the block
consumes.  It performs none of the block's run-time arithmetic (no projection,
score, softmax or requantization of data).
"""

from .generate import (  # noqa: F401
    CONFIGS,
    Block,
    Conv,
    Ffn,
    Residual,
    Workload,
    config_by_name,
    make_block,
    make_conv,
    make_ffn,
    make_residual,
    make_workload,
    sinusoid_table,
)
