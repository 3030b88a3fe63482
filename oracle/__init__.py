"""CPU oracle for the FASQ product-quantized matmul.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library or its binding.
"""

from .pq_oracle import (  # noqa: F401
    lut_accumulate,
    max_abs_over_rms,
    pq_linear,
    reconstruct,
    reconstruct_bits,
    relative_l2,
    unpack_indices,
)
from . import paper_accounting  # noqa: F401
