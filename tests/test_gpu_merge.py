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


# two adapters on q, k, v, o (ranks 16), three sequences
W2 = synth.Workload(name="switch", seed=36, n_layers=3, d_model=512, n_heads=8, d_ffn=1024, vocab=3000,
                    max_pos=64, dtype="f16", batch=3, seq_len=48, lora_targets=("q", "k", "v", "o"),
                    lora_rank=16, lora_alpha=32.0, n_adapters=2, adapter_of_seq=(0, 1, -1))


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _shadow_model(w):
    from paper_2503_17707_amd import binding as pb

    cfg = pb.make_config(w, merge_shadow=True)
    hw = pb.HostWeights(w, cfg)
    m = pb.Model(cfg, "cuda:0")
    pb.attach_all(m, hw)
    m.stream_layers(hw, w.order())
    return hw, m


def test_switching_merged_adapters_through_the_shadow():
    from paper_2503_17707_amd import binding as pb

    log("case merged adapter switching")
    hw, m = _shadow_model(W2)
    try:
        toks = synth.tokens(W2)
        B = W2.batch
        _, base = m.prefill(toks, [-1] * B)
        unmerged = {a: m.prefill(toks, [a] * B) for a in (0, 1)}
        for a in (0, 1, 0):  # merge 0, switch to 1, switch back to 0
            m.merge_lora(a)
            tok, lg = m.prefill(toks, [-1] * B)
            d = float(np.max(np.abs(lg - unmerged[a][1])))
            log("  merged %d vs unmerged: max|d| %.2e" % (a, d))
            assert np.array_equal(tok, unmerged[a][0]) and d <= 2e-2
        first0 = lg
        m.unmerge_lora()
        _, back = m.prefill(toks, [-1] * B)
        assert np.array_equal(_bits(back), _bits(base))  # the shadow restores the base exactly
        with pytest.raises(pb.PbError) as e:
            m.unmerge_lora()
        assert e.value.code == pb.PB_ESTATE
        # a switch gives the bits of a merge onto freshly streamed weights
        m.merge_lora(1)
        m.merge_lora(0)
        _, switched = m.prefill(toks, [-1] * B)
        assert np.array_equal(_bits(switched), _bits(first0))
        pb.attach_all(m, hw)
        m.stream_layers(hw, W2.order())
        m.merge_lora(0)
        _, fresh = m.prefill(toks, [-1] * B)
        assert np.array_equal(_bits(fresh), _bits(first0))
    finally:
        m.destroy()
        hw.free()


def test_epoch_scheduler_serves_a_request_stream_with_merged_adapters():
    """Requests for adapters 0, 1 and the base (a switch with probability 0.2
    between consecutive requests) go through the epoch scheduler; each batch
    runs on the merged model of its adapter, merging or unmerging at the
    switches the scheduler reports, and every request's first token and
    logits equal its unmerged run (bf16: tokens compared where the unmerged
    top-2 margin exceeds the logit tolerance)."""
    from paper_2503_17707_amd import binding as pb

    rng = np.random.default_rng(5)
    n_req = 18
    w = W2.with_(dtype="bf16")
    pool = synth.tokens(w.with_(batch=n_req, seed=77))  # one prompt per request
    adapters, a = [], 0
    for _ in range(n_req):
        if rng.random() < 0.2:
            a = int(rng.choice([x for x in (-1, 0, 1) if x != a]))
        adapters.append(a)
    hw, m = _shadow_model(w)
    s = pb.Scheduler(n_adapters=2, epoch_batches=2)
    try:
        ref = {}
        for i in range(0, n_req, w.batch):  # unmerged reference, the same batch size
            ids = list(range(i, min(i + w.batch, n_req)))
            t, lg = m.prefill(pool[ids], [adapters[j] for j in ids])
            for k, j in enumerate(ids):
                ref[j] = (t[k], lg[k])
        for j in range(n_req):
            s.submit(j, adapters[j])
        merged, served, batches = -1, [], 0
        while True:
            b = s.next(w.batch)
            if b is None:
                break
            ids, a, switched = b
            if switched and a != merged:
                if a >= 0:
                    m.merge_lora(a)
                else:
                    m.unmerge_lora()
                merged = a
            t, lg = m.prefill(pool[ids], [-1] * len(ids))
            for k, j in enumerate(ids):
                assert adapters[j] == a
                top2 = np.sort(ref[j][1])[-2:]
                if top2[1] - top2[0] > 3e-2:
                    assert t[k] == ref[j][0], "request %d: token differs" % j
                assert float(np.max(np.abs(lg[k] - ref[j][1]))) <= 3e-2
            served += ids
            batches += 1
        assert sorted(served) == list(range(n_req))
        log("  %d requests in %d batches, %d switches" % (n_req, batches, s.stats()[1]))
    finally:
        s.close()
        m.destroy()
        hw.free()
