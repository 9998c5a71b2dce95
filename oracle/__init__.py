"""Oracle for the LM operator's row evaluation.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this package.  The library never
calls it and shares no code with it.
"""
from .lmop_oracle import (  # noqa: F401
    KIND_BOOL,
    KIND_ENUM,
    KIND_INT,
    OracleLM,
    attention,
    constrained_pick,
    decode_nibbles,
    dequant,
    rms_norm,
    rope,
    silu,
)
