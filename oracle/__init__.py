"""CPU oracle of the text-encoder prefill (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package; the HIP product path never imports it.
"""
from .te_oracle import (  # noqa: F401
    positions, inv_freq, pair_axis, mrope, rmsnorm, silu, causal_attention,
    layer_forward, encode,
)
