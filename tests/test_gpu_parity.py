"""HIP path vs the CPU oracle, through the C ABI (element by element on the
last-position logits, bit-exact greedy tokens)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import MAX_ABS, compare, log, run_gpu
from storage_rounding import storage_rounded_logits

pytestmark = pytest.mark.gpu

# Small workloads spanning several GEMM tiles, several attention key blocks,
# ragged tails, both head sizes, both storage types and mixed adapters.
SMALL = {
    # the tiny decoder: oracle on the float32 draws, GPU on their bf16 rounding
    "tiny": synth.WORKLOADS["tiny"],
    # three sequences, ragged T, adapters 0 / none / 1 on all four projections
    "mixed": synth.Workload(name="mixed", seed=31, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                            vocab=1000, max_pos=128, dtype="f16", batch=3, seq_len=37,
                            lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                            n_adapters=2, adapter_of_seq=(0, -1, 1)),
    # head_dim 128, bf16, T = 200 (four key blocks, ragged last block)
    "hd128": synth.Workload(name="hd128", seed=32, n_layers=2, d_model=256, n_heads=2, d_ffn=384,
                            vocab=777, max_pos=256, dtype="bf16", batch=2, seq_len=200,
                            lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0, n_adapters=1,
                            oracle_weights="f32"),
    # rank 32 on q, k, v, o, rotated load order, T = max_pos
    "rot": synth.Workload(name="rot", seed=33, n_layers=3, d_model=512, n_heads=8, d_ffn=1024,
                          vocab=3000, max_pos=130, dtype="f16", batch=1, seq_len=130,
                          lora_targets=("q", "k", "v", "o"), lora_rank=32, lora_alpha=64.0,
                          n_adapters=1, layer_order=(2, 0, 1)),
    # every adapter slot the library has (16), one per sequence, on all four
    # projections: the packed LoRA width is 16 x 8 = 128 columns
    "slots16": synth.Workload(name="slots16", seed=37, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                              vocab=900, max_pos=32, dtype="bf16", batch=16, seq_len=20,
                              lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                              n_adapters=16, adapter_of_seq=tuple(range(16))),
    # a single token per sequence and no adapters at all
    "one_token": synth.Workload(name="one_token", seed=34, n_layers=2, d_model=128, n_heads=2,
                                d_ffn=256, vocab=500, max_pos=8, dtype="f16", batch=4, seq_len=1,
                                lora_targets=("q", "v"), lora_rank=4, lora_alpha=8.0,
                                n_adapters=0),
    # eight one-token sequences: every product of the prefill takes the GEMV
    # path with its widest row group (8 rows), adapters mixed on all four
    "eight_tokens": synth.Workload(name="eight_tokens", seed=36, n_layers=2, d_model=256, n_heads=4,
                                   d_ffn=512, vocab=600, max_pos=8, dtype="f16", batch=8, seq_len=1,
                                   lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                                   n_adapters=2, adapter_of_seq=(0, -1, 1, 1, 0, -1, -1, 0)),
    # the largest LoRA rank the library accepts (64), two adapters on all four
    # projections: 128 packed columns, four 16-rank groups per row shrink
    "rank64": synth.Workload(name="rank64", seed=40, n_layers=2, d_model=256, n_heads=4, d_ffn=512,
                             vocab=700, max_pos=64, dtype="bf16", batch=3, seq_len=40,
                             lora_targets=("q", "k", "v", "o"), lora_rank=64, lora_alpha=128.0,
                             n_adapters=2, adapter_of_seq=(1, 0, -1)),
    # the widest model the library accepts (d_model 16384, 128 heads of 128):
    # LayerNorm rows of 16 chunks per thread, the LM head's widest rows (one
    # sequence per launch, three launches), K = 16384 GEMM tiles
    "widest": synth.Workload(name="widest", seed=39, n_layers=1, d_model=16384, n_heads=128,
                             d_ffn=256, vocab=600, max_pos=16, dtype="f16", batch=3, seq_len=9,
                             lora_targets=("q", "v"), lora_rank=4, lora_alpha=8.0, n_adapters=1,
                             adapter_of_seq=(0, -1, 0)),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_workload_matches_oracle(name):
    w = SMALL[name]
    log("case", name, w)
    ref_logits, ref_tok = oracle.prefill_first_token(w)
    tok, logits = run_gpu(w)
    compare(name, logits, tok, ref_logits, ref_tok)


# bf16 storage at the four wider LM-head row lengths (2, 3, 5 and 8 16-byte
# chunks per thread), with 4, 2 + 1, 2 + 1 and 1 + 1 sequences per launch, and
# bf16 LayerNorm, GEMM and head_dim-128 attention at those widths
WIDE_BF16 = {
    "bf16_d4096": synth.Workload(name="bf16_d4096", seed=41, n_layers=1, d_model=4096, n_heads=32,
                                 d_ffn=256, vocab=650, max_pos=16, dtype="bf16", batch=4, seq_len=11,
                                 lora_targets=("q", "k", "v", "o"), lora_rank=8, lora_alpha=16.0,
                                 n_adapters=2, adapter_of_seq=(1, 0, -1, 1)),
    "bf16_d5120": synth.Workload(name="bf16_d5120", seed=42, n_layers=1, d_model=5120, n_heads=40,
                                 d_ffn=256, vocab=620, max_pos=16, dtype="bf16", batch=3, seq_len=10,
                                 lora_targets=("q", "k", "v", "o"), lora_rank=32, lora_alpha=64.0,
                                 n_adapters=1, adapter_of_seq=(0, 0, -1)),
    "bf16_d9216": synth.Workload(name="bf16_d9216", seed=43, n_layers=1, d_model=9216, n_heads=72,
                                 d_ffn=256, vocab=610, max_pos=16, dtype="bf16", batch=3, seq_len=9,
                                 lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0, n_adapters=1,
                                 adapter_of_seq=(0, -1, 0)),
    "bf16_widest": synth.Workload(name="bf16_widest", seed=44, n_layers=1, d_model=16384, n_heads=128,
                                  d_ffn=256, vocab=600, max_pos=16, dtype="bf16", batch=2, seq_len=7,
                                  lora_targets=("q", "v"), lora_rank=4, lora_alpha=8.0, n_adapters=1,
                                  adapter_of_seq=(0, -1)),
}


@pytest.mark.parametrize("name", list(WIDE_BF16))
def test_wide_bf16_matches_oracle_to_storage_rounding(name):
    """Beyond the specified workloads' widths, bf16 activations alone move the
    logits by more than the 3e-2 bar: a float32 CPU build that rounds its
    activations to bf16 where the GPU path stores them misses the oracle by
    2.3e-2 (d_model 4096) to 5.9e-2 (16384), with relative L2 near 5e-3. Here
    the bar on the largest difference is 1.25 times that build's difference
    (never below 3e-2); the relative L2 bar and exact tokens stay as they are."""
    w = WIDE_BF16[name]
    log("case", name, w)
    ref_logits, ref_tok = oracle.prefill_first_token(w)
    storage_err = float(np.max(np.abs(storage_rounded_logits(w, "bf16") - ref_logits)))
    bar = max(MAX_ABS, 1.25 * storage_err)
    log("%s: bf16 storage alone: max|d| %.3e, bar %.3e" % (name, storage_err, bar))
    tok, logits = run_gpu(w)
    compare(name, logits, tok, ref_logits, ref_tok, max_abs=bar)


def test_tiny_storage_rounding_and_kernel_error_apart():
    """The tiny decoder's oracle runs on the float32 draws while the GPU stores
    their bf16 rounding; the oracle on the bf16-widened weights isolates the
    kernels' own error from that storage rounding.  Both are logged, both are
    within tolerance."""
    w = SMALL["tiny"]
    log("case tiny: storage rounding vs kernel error")
    tok, logits = run_gpu(w)
    ref32, tok32 = oracle.prefill_first_token(w)
    ref16, tok16 = oracle.prefill_first_token(w.with_(oracle_weights="storage"))
    d32 = compare("tiny vs oracle on f32 draws", logits, tok, ref32, tok32)
    d16 = compare("tiny vs oracle on bf16 weights", logits, tok, ref16, tok16)
    log("  storage + kernel max|d| %.2e, kernel alone %.2e" % (d32[0], d16[0]))


def test_lora_with_zero_b_is_bit_identical_to_base():
    w = SMALL["mixed"].with_(lora_zero_b=True)
    log("case lora_zero_b")
    tok_a, log_a = run_gpu(w, adapters=(0, 1, 1))
    tok_b, log_b = run_gpu(w, adapters=(-1, -1, -1))
    assert np.array_equal(log_a.view(np.uint32), log_b.view(np.uint32))
    assert np.array_equal(tok_a, tok_b)


def test_reorder_invariance_is_bit_exact():
    from paper_2503_17707_amd import binding as pb

    w = SMALL["rot"].with_(n_layers=6, layer_order=None)
    log("case reorder")
    hw, m0 = pb.setup(w)
    m0.destroy()
    orders = [list(range(6)), list(range(5, -1, -1)), [3, 4, 5, 0, 1, 2], [4, 1, 5, 0, 2, 3]]
    outs = []
    try:
        for o in orders:
            tok, logits = run_gpu(w, order=o, hw=hw)
            outs.append((tok, logits))
    finally:
        hw.free()
    for tok, logits in outs[1:]:
        assert np.array_equal(tok, outs[0][0])
        assert np.array_equal(logits.view(np.uint32), outs[0][1].view(np.uint32))


def test_repeat_runs_are_bit_identical_and_warm_prefill_matches_cold():
    from paper_2503_17707_amd import binding as pb

    w = SMALL["mixed"]
    log("case determinism")
    hw, m = pb.setup(w)
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw)
        toks = synth.tokens(w)
        t1, l1 = m.prefill(toks, w.adapters())
        t2, l2 = m.prefill(toks, w.adapters())  # warm: weights resident
        assert np.array_equal(t1, t2)
        assert np.array_equal(l1.view(np.uint32), l2.view(np.uint32))
    finally:
        m.destroy()
        hw.free()


def test_poisoned_weights_and_late_copies_never_leak():
    """NaN-poison the device weights, then make the host enqueue each layer's
    copies late: any kernel that ran before its layer landed would read NaN."""
    from paper_2503_17707_amd import binding as pb

    w = SMALL["rot"]
    log("case poison")
    hw, m = pb.setup(w)
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw, w.order())
        toks = synth.tokens(w)
        ref_tok, ref = m.prefill(toks, w.adapters())
        for delay in (0, 20000):
            m.poison(0xFF)
            m.set_stream_delay_us(delay)
            pb.attach_all(m, hw)
            m.stream_layers(hw, w.order())
            tok, logits = m.prefill(toks, w.adapters())
            assert np.all(np.isfinite(logits))
            assert np.array_equal(tok, ref_tok)
            assert np.array_equal(logits.view(np.uint32), ref.view(np.uint32))
    finally:
        m.destroy()
        hw.free()


def test_pageable_layer_blobs_are_staged_bitwise():
    """Layer blobs in pageable host memory go through the loader's pinned
    staging ring on its own thread: all-pageable and half-pinned loads, with
    poisoned device weights and late enqueues, give bit-identical results to
    an all-pinned load."""
    from paper_2503_17707_amd import binding as pb

    w = SMALL["rot"]
    log("case pageable layer blobs")
    cfg = pb.make_config(w)
    hw, m = pb.setup(w)
    hws = [pb.HostWeights(w, cfg, pin_budget=0),
           pb.HostWeights(w, cfg, pin_budget=(w.n_layers // 2) * hw.layer_bytes)]
    try:
        for h in [hw] + hws:
            for a in sorted({a for a in w.adapters() if a >= 0}):
                h.add_lora(a)
        assert hws[0].pinned_layers == 0 and 0 < hws[1].pinned_layers < w.n_layers
        toks = synth.tokens(w)
        pb.attach_all(m, hw)
        m.stream_layers(hw, w.order())
        ref_tok, ref = m.prefill(toks, w.adapters())
        for h in hws:
            for delay in (0, 20000):
                m.poison(0xFF)
                m.set_stream_delay_us(delay)
                pb.attach_all(m, h)
                m.stream_layers(h, w.order())
                tok, logits = m.prefill(toks, w.adapters())
                nbytes, ms = m.load_stats()
                log("  pinned layers %d/%d, delay %d us: load %.2f ms" % (
                    h.pinned_layers, w.n_layers, delay, ms))
                assert nbytes > 0 and ms > 0
                assert np.array_equal(tok, ref_tok)
                assert np.array_equal(logits.view(np.uint32), ref.view(np.uint32))
        m.set_stream_delay_us(0)
    finally:
        m.destroy()
        for h in [hw] + hws:
            h.free()


def test_mixed_batch_equals_each_sequence_alone():
    """Per-sequence adapter gather: a mixed batch gives each sequence the
    result it gets alone (up to the batch's own reduction orders: exact here,
    since rows never interact)."""
    from paper_2503_17707_amd import binding as pb

    w = SMALL["mixed"]
    log("case per-sequence adapters")
    hw, m = pb.setup(w)
    try:
        pb.attach_all(m, hw)
        m.stream_layers(hw)
        toks = synth.tokens(w)
        tok, logits = m.prefill(toks, w.adapters())
        for b, a in enumerate(w.adapters()):
            t1, l1 = m.prefill(toks[b:b + 1], [a])
            assert t1[0] == tok[b]
            assert np.max(np.abs(l1[0] - logits[b])) <= 1e-5
    finally:
        m.destroy()
        hw.free()
