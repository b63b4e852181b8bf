"""CPU oracle for the 4-bit group-quantized decode linears.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .wq_oracle import (  # noqa: F401
    ABS_TOL,
    GROUP,
    REL_TOL,
    dequant,
    gemv,
    gemv_f64,
    quantize_pack,
    tol_bound,
    unpack,
    within_tolerance,
)
from .attn_oracle import (  # noqa: F401
    ATTN_ABS_TOL,
    ATTN_MAX_SCORE_BOUND,
    ATTN_REL_TOL,
    attn_tol_bound,
    attn_within_tolerance,
    decode_attention,
    decode_attention_f64,
)
