"""Pins of the storage-rounding model (tests/storage_rounding.py) on the CPU.

That model sets the logit bar of the GPU parity cases with bf16 storage at
widths beyond the specified workloads. Here it is checked against the float64
oracle:
- without rounding it is the oracle's decoder in float32 arithmetic;
- with rounding its error grows by the storage dtype's precision, bf16's
  8 significant bits against fp16's 11.
"""
import numpy as np
import pytest

import oracle
import synth
from storage_rounding import storage_rounded_logits

# LoRA on all four projections, two adapters and a sequence without one, so
# that every branch of the model runs
MINI = synth.Workload(name="mini-sr", seed=111, n_layers=2, d_model=64, n_heads=4, d_ffn=128,
                      vocab=97, max_pos=16, dtype="bf16", batch=3, seq_len=7,
                      lora_targets=("q", "k", "v", "o"), lora_rank=4, lora_alpha=8.0,
                      n_adapters=2, adapter_of_seq=(0, -1, 1))
# wide enough that the activations' rounding shows well above float32's
WIDE = synth.Workload(name="wide-sr", seed=112, n_layers=1, d_model=512, n_heads=4, d_ffn=256,
                      vocab=300, max_pos=16, dtype="bf16", batch=2, seq_len=9,
                      lora_targets=("q", "v"), lora_rank=8, lora_alpha=16.0, n_adapters=1,
                      adapter_of_seq=(0, -1))


def _rel(got, ref):
    return float(np.max(np.linalg.norm(got - ref, axis=-1) / np.linalg.norm(ref, axis=-1)))


@pytest.mark.parametrize("w", [MINI, MINI.with_(name="mini-sr-f16", dtype="f16"), WIDE],
                         ids=["mini-bf16", "mini-f16", "wide-bf16"])
def test_without_rounding_it_is_the_oracle_in_float32(w):
    ref, _ = oracle.prefill_first_token(w)
    got = storage_rounded_logits(w, None)
    assert _rel(got, ref) < 1e-5
    assert np.max(np.abs(got - ref)) < 1e-4 * max(1.0, np.max(np.abs(ref)))


def test_rounding_error_follows_the_storage_precision():
    ref, _ = oracle.prefill_first_token(WIDE)
    e32 = _rel(storage_rounded_logits(WIDE, None), ref)
    e16 = _rel(storage_rounded_logits(WIDE, "f16"), ref)
    eb16 = _rel(storage_rounded_logits(WIDE, "bf16"), ref)
    # each rounding is relative 2^-9 (bf16) or 2^-12 (fp16) at most: the errors
    # stand well above float32's and bf16's about eight times fp16's
    assert e32 < 1e-5 < e16 < eb16 < 1e-2
    assert 3.0 < eb16 / e16 < 20.0
