"""Pipeline stages on one GPU (Sections 4.2.1, 4.3.1): models that each hold
a contiguous block of layers (streamed as a partial layer order) run their
block and hand the fp32 hidden states on; the last stage returns the first
tokens.  Every stage runs the kernels a full prefill would run on its layers,
so the chain must reproduce one full prefill bit for bit."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_common import compare, golden_path, log

pytestmark = pytest.mark.gpu

# four layers, two adapters and the base mixed in one batch, rank 16 on q, k, v, o
W = synth.Workload(name="stages", seed=38, n_layers=4, d_model=256, n_heads=4, d_ffn=512, vocab=1000,
                   max_pos=64, dtype="f16", batch=3, seq_len=45, lora_targets=("q", "k", "v", "o"),
                   lora_rank=16, lora_alpha=32.0, n_adapters=2, adapter_of_seq=(1, -1, 0))


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _stage_model(pb, hw, order):
    m = pb.Model(pb.make_config(W), "cuda:0")
    pb.attach_all(m, hw)
    m.stream_layers(hw, order)
    return m


@pytest.mark.parametrize("blocks", [[(0, 2), (2, 4)], [(0, 1), (1, 3), (3, 4)]])
def test_stage_chain_equals_full_prefill(blocks):
    import torch
    from paper_2503_17707_amd import binding as pb

    log("case stages", blocks)
    cfg = pb.make_config(W)
    hw = pb.HostWeights(W, cfg)
    full = pb.Model(cfg, "cuda:0")
    models = []
    try:
        pb.attach_all(full, hw)
        full.stream_layers(hw)
        toks = synth.tokens(W)
        ad = list(W.adapters())
        ref_tok, ref = full.prefill(toks, ad)
        # each stage streams only its own block, in reverse order for good measure
        models = [_stage_model(pb, hw, list(range(b, e))[::-1]) for b, e in blocks]
        hid = torch.empty(W.batch * W.seq_len, W.d_model, dtype=torch.float32, device="cuda:0")
        out = None
        for (b, e), m in zip(blocks, models):
            out = m.prefill_stage(toks, ad, b, e, hidden_in=hid if b > 0 else None,
                                  hidden_out=hid if e < W.n_layers else None)
        tok, lg = out
        # the chain against the oracle's prefill of the same workload
        o_logits, o_tok = oracle.prefill_first_token(W, tokens=toks, adapter_of_seq=ad)
        compare("stages %s" % blocks, lg, tok, o_logits, o_tok)
        assert np.array_equal(tok, ref_tok)
        assert np.array_equal(_bits(lg), _bits(ref))
        # a stage on a model that lacks one of its layers fails cleanly
        with pytest.raises(pb.PbError) as e:
            models[0].prefill_stage(toks, ad, 0, W.n_layers)
        assert e.value.code == pb.PB_ESTATE
    finally:
        for m in models + [full]:
            m.destroy()
        hw.free()


def test_stage_cold_start_waits_for_its_own_layers():
    """A stage enqueued right after its (poisoned, late) partial load still
    reads only landed weights."""
    import torch
    from paper_2503_17707_amd import binding as pb

    cfg = pb.make_config(W)
    hw = pb.HostWeights(W, cfg)
    a = b = None
    try:
        toks = synth.tokens(W)
        ad = list(W.adapters())
        a = _stage_model(pb, hw, [0, 1])
        b = _stage_model(pb, hw, [3, 2])
        hid = torch.empty(W.batch * W.seq_len, W.d_model, dtype=torch.float32, device="cuda:0")
        a.prefill_stage(toks, ad, 0, 2, hidden_out=hid)
        ref_tok, ref = b.prefill_stage(toks, ad, 2, 4, hidden_in=hid)
        for m, order in ((a, [1, 0]), (b, [2, 3])):
            m.poison(0xFF)
            m.set_stream_delay_us(5000)
            pb.attach_all(m, hw)
            m.stream_layers(hw, order)
        a.prefill_stage(toks, ad, 0, 2, hidden_out=hid)
        tok, lg = b.prefill_stage(toks, ad, 2, 4, hidden_in=hid)
        assert np.all(np.isfinite(lg))
        assert np.array_equal(tok, ref_tok) and np.array_equal(_bits(lg), _bits(ref))
    finally:
        for m in (a, b):
            if m is not None:
                m.destroy()
        hw.free()


def test_stage_argument_errors():
    from paper_2503_17707_amd import binding as pb

    cfg = pb.make_config(W)
    hw = pb.HostWeights(W, cfg)
    m = _stage_model(pb, hw, [0, 1, 2, 3])
    try:
        toks = synth.tokens(W)
        ad = list(W.adapters())
        for lb, le in ((2, 2), (-1, 2), (0, 5), (3, 1)):
            with pytest.raises(pb.PbError) as e:
                m.prefill_stage(toks, ad, lb, le)
            assert e.value.code == pb.PB_EINVAL, (lb, le)
        with pytest.raises(pb.PbError) as e:  # a later stage without its input
            m.prefill_stage(toks, ad, 2, 4)
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:  # an earlier stage without its output
            m.prefill_stage(toks, ad, 0, 2)
        assert e.value.code == pb.PB_EINVAL
    finally:
        m.destroy()
        hw.free()


def test_opt1_3b_two_stage_split_matches_oracle():
    """OPT-1.3B (24 layers, 512 tokens, LoRA r16 on q,v) run as two stages of
    one GPU's share: layers 0-11 on one model, 12-23 on another, each loading
    only its own block; the first token and logits against the oracle's stored
    logits for the whole model."""
    import torch
    from paper_2503_17707_amd import binding as pb

    name = "opt-1.3b"
    p = golden_path(name)
    if not os.path.exists(p):
        pytest.skip("oracle logits for %s not generated" % name)
    g = np.load(p, allow_pickle=False)
    w = synth.WORKLOADS[name]
    log("case stages opt-1.3b 0-11 | 12-23")
    cfg = pb.make_config(w)
    hw = pb.HostWeights(w, cfg)
    models = []
    try:
        half = w.n_layers // 2
        for blk in (range(0, half), range(half, w.n_layers)):
            m = pb.Model(cfg, "cuda:0")
            models.append(m)
            pb.attach_all(m, hw)
            m.stream_layers(hw, list(blk))
        toks = synth.tokens(w)
        ad = list(w.adapters())
        hid = torch.empty(w.n_tokens, w.d_model, dtype=torch.float32, device="cuda:0")
        models[0].prefill_stage(toks, ad, 0, half, hidden_out=hid)
        tok, lg = models[1].prefill_stage(toks, ad, half, w.n_layers, hidden_in=hid)
        compare("stages opt-1.3b", lg, tok, g["logits"], g["tokens"])
    finally:
        for m in models:
            m.destroy()
        hw.free()
