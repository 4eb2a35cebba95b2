"""Float64 CPU oracle for composed-KV attention (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path never calls it; it shares no code with
the HIP library or its Python binding.
"""
from .c2kv_oracle import (  # noqa: F401
    decode_bf16, decode_storage, rope_theta, rope_rotate, compose_layout,
    compose, attend, compose_attend, merge_partials, sif_positions, sif_mask, sif_attend,
)
