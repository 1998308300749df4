"""QEvict tiered decode step for MI355X (gfx950): HIP kernels behind a C ABI.

The library (libqevict.so, built from csrc/ by ``build.py``) implements the
per-step hot path of QEvict (arXiv 2608.05326): split-K decode attention over
bf16 and quantized windows with per-window mass accumulation, TopK re-tiering
and the quantize / promote migrations.  ``qevict`` is the ctypes binding.
"""
from .qevict import (  # noqa: F401
    Cache, Config, QEvictError, RetierStats, load_library, workspace_size, SYMBOLS,
    OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_BAD_STATE, ERR_NONFINITE,
    ERR_CAPACITY, ERR_DEVICE,
    TIER_UNUSED, TIER_OPEN, TIER_FULL, TIER_QUANT, TIER_EVICTED,
    LEDGER_NONE, LEDGER_ACTIVE, LEDGER_DORMANT, BITS_MIXED_4_2, OUT_F32, OUT_BF16,
    FLAG_NO_PROMOTION, FLAG_DEBUG_MASSES, FLAG_ASYNC_ROUTING, FLAG_ROUTING_QUEUE_WAIT,
    FLAG_ROUTING_DEVICE_WAIT,
    KERNEL_ATTEND, KERNEL_MERGE, KERNEL_RETIER, KERNEL_MIGRATE, SCORE_CUMULATIVE, SCORE_DECAY, SCORE_KEY_NORM,
    SCORE_PNORM,
)
