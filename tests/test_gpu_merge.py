"""Merged LoRA (Section 4.3.2): the adapter folded into the device base
weights gives the model the oracle computes with the adapter unmerged (the two
agree in exact arithmetic; here up to the one rounding of the merged weights),
with no LoRA work left on the hot path."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import compare, log

pytestmark = pytest.mark.gpu

# rank 32 on q, k, v, o, one adapter for the single sequence
W = synth.Workload(name="merge", seed=35, n_layers=3, d_model=512, n_heads=8, d_ffn=1024, vocab=3000,
                   max_pos=130, dtype="f16", batch=1, seq_len=130, lora_targets=("q", "k", "v", "o"),
                   lora_rank=32, lora_alpha=64.0, n_adapters=1, layer_order=(2, 0, 1))


def test_merged_lora_matches_oracle_and_unmerged():
    from paper_2503_17707_amd import binding as pb

    log("case merged lora")
    hw, m = pb.setup(W)
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw, W.order())
        toks = synth.tokens(W)
        base_tok, base = m.prefill(toks, [-1])
        tok_u, log_u = m.prefill(toks, [0])
        m.merge_lora(0)
        with pytest.raises(pb.PbError) as e:  # the adapter is part of the base now
            m.prefill(toks, [0])
        assert e.value.code == pb.PB_ESTATE
        with pytest.raises(pb.PbError) as e:  # merging twice would apply it twice
            m.merge_lora(0)
        assert e.value.code == pb.PB_ESTATE
        tok_m, log_m = m.prefill(toks, [-1])
        ref, ref_tok = oracle.prefill_first_token(W, adapter_of_seq=[0])
        compare("merged vs oracle (unmerged adapter)", log_m, tok_m, ref, ref_tok)
        d = float(np.max(np.abs(log_m - log_u)))
        log("  merged vs unmerged on the GPU: max|d| %.2e" % d)
        assert np.array_equal(tok_m, tok_u) and d <= 2e-2
        # streaming the base again undoes the merge exactly
        pb.attach_all(m, hw)
        m.stream_layers(hw, W.order())
        tok_b, log_b = m.prefill(toks, [-1])
        assert np.array_equal(log_b.view(np.uint32), base.view(np.uint32))
        assert np.array_equal(tok_b, base_tok)
    finally:
        m.destroy()
        hw.free()


def test_merging_a_zero_b_adapter_leaves_the_base_bit_identical():
    from paper_2503_17707_amd import binding as pb

    w = W.with_(lora_zero_b=True)
    hw, m = pb.setup(w)
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw, w.order())
        toks = synth.tokens(w)
        _, base = m.prefill(toks, [-1])
        m.merge_lora(0)
        _, merged = m.prefill(toks, [-1])
        assert np.array_equal(merged.view(np.uint32), base.view(np.uint32))
    finally:
        m.destroy()
        hw.free()
