"""CPU oracle for the Gated DeltaNet decode / prefill path (fp64, token by token).

TEST INFRASTRUCTURE ONLY: imported by tests, by the smoke check and by the
benchmark's CPU-baseline leg.  The HIP library and its Python binding never
import it.  See gdn_ref.py for what is computed and the passages it follows.
"""
from .gdn_ref import (  # noqa: F401
    GATE_LOGITS,
    QK_L2NORM,
    bf16_rne_bits,
    decode,
    gate_from_logits,
    head_map,
    prefill_chunked,
    prefill_transfer,
    prefill_units,
    prefill_varlen,
    prologue,
    qk_l2norm_bf16,
    step_matrix,
    step_rank1,
    to_f64,
)
