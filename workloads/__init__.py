"""Seeded synthetic workloads for the mixed prefill/decode paged-attention step.

This package only draws inputs: batch metadata (rows, block tables, pool
sizes), the config-5 scheduler replay that produces such metadata, and the
bf16 tensors.  It holds none of the attention arithmetic, so both the fp64
oracle and the HIP library can consume what it produces without sharing any
of the method's code.
"""

from .configs import (  # noqa: F401
    Batch,
    CONFIG_NAMES,
    make_batch,
    make_config,
    replay_schedule,
    subset,
    tiny_batch,
)
from .tensors import make_caches, make_step_tensors, make_tensors  # noqa: F401
from .serving import short_long_stream, uniform_stream  # noqa: F401
