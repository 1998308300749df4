"""Plain float64 CPU oracle of the QEvict decode step.

TEST INFRASTRUCTURE: imported only by tests, the smoke check and the
benchmark's CPU-baseline leg.  It shares no code with the GPU library.
"""
from .numerics import rne_bf16, rne_fp16, rd_fp16, ru_fp16  # noqa: F401
from .qevict_oracle import (  # noqa: F401
    OPEN, AGED, FULL, QUANT, EVICTED, ACTIVE, DORMANT,
    OracleConfig, QEvictUnit, quantize_groups, quantize_window, dequantize_window,
    route_order, tier_split,
)
