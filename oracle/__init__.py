"""CPU oracle for the cold-start prefill path (test infrastructure only).

Only the tests, the package's ``smoke()`` check and the benchmark's CPU
baseline may import this package.  The GPU path never calls it, links it or
falls back to it.
"""
from .opt_lora import (  # noqa: F401
    attention_weights,
    causal_self_attention,
    decoder_layer,
    final_logits,
    greedy_token,
    layer_norm,
    lora_delta,
    prefill_first_token,
    widen,
    WeightSource,
)
