"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds no arithmetic of the pruning method: it only draws
tensors (fp32, optionally rounded to bf16 bit patterns) and describes the
layer shapes of the workloads.  Both the oracle and the HIP path consume
the exact same host bits produced here.
"""

from .gen import (  # noqa: F401
    SEED_X, SEED_W, SEED_B, seed_for, f32_to_bf16_bits, bf16_bits_to_f32,
    draw, draw_layer, draw_device,
)
from .workloads import (  # noqa: F401
    Scheme, ConvLayer, LinearLayer, workload, WORKLOADS,
    ROW, COL, UNSTRUCTURED, DENSE, PUNCHED, ROWCOL, PATTERN,
)
