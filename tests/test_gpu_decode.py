"""Decode steps with the KV cache against the oracle: the greedy token and the
logits of step k are those of a plain prefill over the prompt plus the k
tokens generated so far (the decode stage of Section 2.1 computes exactly
that, reusing the cached keys and values)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import compare, log

pytestmark = pytest.mark.gpu

CASES = {
    # three sequences, adapters 0 / none / 1 on q, k, v, o, f16, head_dim 64
    "mixed": synth.Workload(name="mixed", seed=31, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                            vocab=1000, max_pos=128, dtype="f16", batch=3, seq_len=37,
                            lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                            n_adapters=2, adapter_of_seq=(0, -1, 1)),
    # bf16, head_dim 128, a prompt longer than one pass of the block's waves
    # over the keys (8 waves x 64 keys)
    "hd128": synth.Workload(name="hd128", seed=32, n_layers=2, d_model=256, n_heads=2, d_ffn=384,
                            vocab=777, max_pos=640, dtype="bf16", batch=2, seq_len=560,
                            lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0, n_adapters=1),
    # f16, head_dim 64, past one pass of 16 waves x 64 keys
    "long64": synth.Workload(name="long64", seed=33, n_layers=2, d_model=128, n_heads=2, d_ffn=256,
                             vocab=500, max_pos=1040, dtype="f16", batch=1, seq_len=1030,
                             lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=8.0, n_adapters=1),
    # f16 with head_dim 128 (the OPT-6.7B to 66B head size and storage type)
    "f16_hd128": synth.Workload(name="f16_hd128", seed=38, n_layers=2, d_model=256, n_heads=2, d_ffn=384,
                                vocab=700, max_pos=96, dtype="f16", batch=2, seq_len=70,
                                lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0, n_adapters=1,
                                adapter_of_seq=(0, -1)),
    # the largest rank (64) on q, k, v, o with two adapters: the decode
    # LayerNorm's shrink spread over 48 blocks of 4 ranks per row
    "rank64": synth.Workload(name="rank64", seed=40, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                             vocab=700, max_pos=48, dtype="bf16", batch=3, seq_len=24,
                             lora_targets=("q", "k", "v", "o"), lora_rank=64, lora_alpha=128.0,
                             n_adapters=2, adapter_of_seq=(1, 0, -1)),
    # six sequences: the GEMVs' widest row group (8 token rows, two of them
    # clamped), three adapters and the base mixed, bf16
    "batch6": synth.Workload(name="batch6", seed=35, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                             vocab=800, max_pos=64, dtype="bf16", batch=6, seq_len=21,
                             lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                             n_adapters=3, adapter_of_seq=(0, 1, -1, 2, 0, -1)),
}
STEPS = 4


def _model(w, new_tokens):
    from paper_2503_17707_amd import binding as pb

    cfg = pb.make_config(w, max_new_tokens=new_tokens)
    hw = pb.HostWeights(w, cfg)
    m = pb.Model(cfg, "cuda:0")
    pb.attach_all(m, hw)
    m.stream_layers(hw, w.order())
    return hw, m


@pytest.mark.parametrize("name", list(CASES))
def test_decode_steps_match_oracle_prefill_of_extended_prompt(name):
    w = CASES[name]
    log("case decode", name)
    hw, m = _model(w, STEPS)
    try:
        ad = list(w.adapters())
        seq = synth.tokens(w).astype(np.int32)
        tok, logits = m.prefill(seq, ad)
        for step in range(STEPS):
            seq = np.concatenate([seq, tok[:, None]], axis=1)
            tok, logits = m.decode(tok, ad)
            ref_logits, ref_tok = oracle.prefill_first_token(w, tokens=seq, adapter_of_seq=ad)
            compare("%s decode step %d (T=%d)" % (name, step + 1, seq.shape[1]), logits, tok,
                    ref_logits, ref_tok)
    finally:
        m.destroy()
        hw.free()


def test_decode_equals_gpu_prefill_of_extended_prompt():
    """The cached path and a fresh prefill over the longer prompt agree to
    rounding (different reduction orders only)."""
    w = CASES["mixed"]
    hw, m = _model(w, 2)
    try:
        ad = list(w.adapters())
        seq = synth.tokens(w).astype(np.int32)
        tok, _ = m.prefill(seq, ad)
        tok2, dec_logits = m.decode(tok, ad)
        ext = np.concatenate([seq, tok[:, None]], axis=1)
        w2 = w.with_(seq_len=ext.shape[1])
        from paper_2503_17707_amd import binding as pb
        hw2, m2 = pb.setup(w2)
        try:
            pb.attach_all(m2, hw2)
            m2.stream_layers(hw2)
            tok_p, pre_logits = m2.prefill(ext, ad)
        finally:
            m2.destroy()
            hw2.free()
        log("  decode vs prefill max|d| %.2e" % float(np.max(np.abs(dec_logits - pre_logits))))
        assert np.array_equal(tok2, tok_p)
        assert float(np.max(np.abs(dec_logits - pre_logits))) <= 2e-2
    finally:
        m.destroy()
        hw.free()


def test_decode_state_errors():
    from paper_2503_17707_amd import binding as pb

    w = CASES["mixed"]
    ad = list(w.adapters())
    seq = synth.tokens(w).astype(np.int32)
    # no KV cache in the config
    hw, m = _model(w, 0)
    try:
        tok, _ = m.prefill(seq, ad)
        with pytest.raises(pb.PbError) as e:
            m.decode(tok, ad)
        assert e.value.code == pb.PB_ESTATE
    finally:
        m.destroy()
        hw.free()
    hw, m = _model(w, 1)
    try:
        with pytest.raises(pb.PbError) as e:  # nothing to continue yet
            m.decode(seq[:, 0], ad)
        assert e.value.code == pb.PB_ESTATE
        tok, _ = m.prefill(seq, ad)
        with pytest.raises(pb.PbError) as e:  # another batch size
            m.decode(tok[:2], ad[:2])
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:  # another adapter
            m.decode(tok, [1, -1, 1])
        assert e.value.code == pb.PB_EINVAL
        tok, _ = m.decode(tok, ad)
        with pytest.raises(pb.PbError) as e:  # max_new_tokens = 1 reached
            m.decode(tok, ad)
        assert e.value.code == pb.PB_ESTATE
    finally:
        m.destroy()
        hw.free()


def test_opt_1_3b_decode_matches_stored_oracle_steps():
    """OPT-1.3B workload: two greedy decode steps after the cold-start prefill
    against the oracle's stored logits of those steps (make_golden.py --decode)."""
    import os

    from gpu_common import golden_path

    name = "opt-1.3b"
    p = golden_path(name + "-decode")
    if not os.path.exists(p):
        pytest.skip("oracle decode logits for %s not generated" % name)
    g = np.load(p, allow_pickle=False)
    w = synth.WORKLOADS[name]
    k = g["tokens"].shape[0]
    log("case decode", name, "steps", k)
    hw, m = _model(w, k)
    try:
        ad = list(w.adapters())
        tok, _ = m.prefill(synth.tokens(w), ad)
        for i in range(k):
            tok, logits = m.decode(tok, ad)
            compare("%s decode step %d" % (name, i + 1), logits, tok, g["logits"][i].astype(np.float64),
                    g["tokens"][i])
    finally:
        m.destroy()
        hw.free()


@pytest.mark.parametrize("lost", [(0, 1, 0, 1), (1, 1, 1, 1)])
def test_kv_rebuild_after_losing_layers(lost):
    """Failure recovery (Section 4.4.2): after two decode steps the KV cache of
    some layers is lost (NaN-filled).  A rebuild over the tokens processed so
    far recomputes only the queries in the surviving layers and everything in
    the lost ones; it reproduces the last decode output, and decoding then
    continues as the oracle says."""
    w = CASES["mixed"].with_(n_layers=4)
    B, T = w.batch, w.seq_len
    from paper_2503_17707_amd import binding as pb

    log("case kv rebuild, lost layers", lost)
    cfg = pb.make_config(w, max_new_tokens=4, max_tokens=B * (T + 4))
    hw = pb.HostWeights(w, cfg)
    m = pb.Model(cfg, "cuda:0")
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw, w.order())
        ad = list(w.adapters())
        seq = synth.tokens(w).astype(np.int32)
        t1, _ = m.prefill(seq, ad)
        t2, _ = m.decode(t1, ad)
        t3, _ = m.decode(t2, ad)
        processed = np.concatenate([seq, t1[:, None], t2[:, None]], axis=1)
        m.invalidate_kv([bool(x) for x in lost])
        r3, lg3 = m.rebuild_kv(processed, [not x for x in lost], ad)
        assert np.all(np.isfinite(lg3))
        assert np.array_equal(r3, t3)
        ref, ref_tok = oracle.prefill_first_token(w, tokens=processed, adapter_of_seq=ad)
        compare("rebuild (T=%d)" % processed.shape[1], lg3, r3, ref, ref_tok)
        t4, lg4 = m.decode(r3, ad)
        ext = np.concatenate([processed, r3[:, None]], axis=1)
        ref, ref_tok = oracle.prefill_first_token(w, tokens=ext, adapter_of_seq=ad)
        compare("decode after rebuild (T=%d)" % ext.shape[1], lg4, t4, ref, ref_tok)
    finally:
        m.destroy()
        hw.free()
