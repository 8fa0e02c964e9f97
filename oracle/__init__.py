"""CPU oracle for the budget-adapted prefill -- TEST INFRASTRUCTURE ONLY.

Imported only by the test suite, the smoke check and the benchmark's CPU
baseline; never by the product path.  See prefill.py for what it computes.
"""
from .prefill import (
    FlopCounter, PrefillResult, causal_attention, compact, decoder_layer, prefill, rmsnorm,
    rope, select_and_compact, select_topk, silu,
)

__all__ = [
    "FlopCounter", "PrefillResult", "causal_attention", "compact", "decoder_layer", "prefill",
    "rmsnorm", "rope", "select_and_compact", "select_topk", "silu",
]
