"""CPU oracle for the Gated DeltaNet decode / prefill path (fp64, token by token).

TEST INFRASTRUCTURE ONLY: imported by tests, by the smoke check and by the
benchmark's CPU-baseline leg.  The HIP library and its Python binding never
import it.  See gdn_ref.py for what is computed and the passages it follows.
"""
from .gdn_ref import (  # noqa: F401
    decode,
    head_map,
    prefill_chunked,
    prefill_transfer,
    prefill_units,
    prefill_varlen,
    step_matrix,
    step_rank1,
    to_f64,
)
