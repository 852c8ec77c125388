"""CPU oracle for topology-biased graph attention.

TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path (the HIP library
and its Python binding) never does. The oracle shares no code with the HIP
path: both read their inputs from the ``synth`` package, nothing else.

Plain, slow, fp64 NumPy that materialises every score block in full.
"""
from .attention import (  # noqa: F401
    bias_block,
    block_attention,
    block_backward,
    forward,
    backward,
    ring_step,
    merge,
    ring_forward,
    ring_backward_step,
    ring_backward,
    super_shard_rows,
    ring_forward_super,
    ring_backward_super,
    lse_bias_only,
)
