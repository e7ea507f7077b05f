"""Pins of the CPU oracle against facts that do not come from the oracle itself.

* closed forms and invariants of LayerNorm and causal softmax attention;
* brute force on tiny inputs;
* LoRA with B = 0 leaves the base model bit-identical; the unmerged delta
  equals the merged weight W + s B A of the paper's Section 4.3.2;
* causality: tokens after position t cannot change positions <= t;
* an independent float64 build of the whole decoder from torch.nn.functional
  library routines (layer_norm, linear, scaled_dot_product_attention, relu),
  with LoRA merged into the weights per sequence;
* exact widening of stored fp16 / bf16 bit patterns to float64, against
  values fixed by the two formats' definitions;
* planted mistakes in the oracle are caught by these pins.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import oracle.opt_lora as ol
import synth

MINI = synth.Workload(name="mini", seed=101, n_layers=2, d_model=64, n_heads=4, d_ffn=128,
                      vocab=97, max_pos=16, dtype="f16", batch=3, seq_len=7,
                      lora_targets=("q", "k", "v", "o"), lora_rank=4, lora_alpha=8.0,
                      n_adapters=2, adapter_of_seq=(0, -1, 1))
TINY = synth.WORKLOADS["tiny"]
# the same decoder stored in bfloat16 (the tiny workload's GPU storage type)
MINI_BF16 = MINI.with_(name="mini-bf16", dtype="bf16")


# ----------------------------------------------------------------------------
# LayerNorm
# ----------------------------------------------------------------------------

def test_layernorm_moments_before_affine():
    rng = np.random.default_rng(0)
    x = rng.normal(3.0, 2.5, size=(50, 301))
    y = oracle.layer_norm(x, np.ones(301), np.zeros(301), 1e-5)
    var = x.var(axis=1)
    assert np.max(np.abs(y.mean(axis=1))) < 1e-12
    # biased variance of the output is var / (var + eps)
    assert np.allclose(y.var(axis=1), var / (var + 1e-5), rtol=1e-12, atol=0)


def test_layernorm_matches_torch_library():
    rng = np.random.default_rng(1)
    x = rng.normal(0.0, 1.5, size=(17, 96))
    g = rng.normal(1.0, 0.1, size=96)
    b = rng.normal(0.0, 0.1, size=96)
    ref = F.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), torch.from_numpy(b),
                       1e-5).numpy()
    assert np.max(np.abs(oracle.layer_norm(x, g, b, 1e-5) - ref)) < 1e-12


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------

def _brute_attention(q, k, v):
    T, hd = q.shape
    out = np.zeros_like(v)
    for j in range(T):
        scores = [sum(q[j, c] * k[i, c] for c in range(hd)) for i in range(j + 1)]
        m = max(scores)
        e = [math.exp(s - m) for s in scores]
        z = sum(e)
        for c in range(v.shape[1]):
            out[j, c] = sum(e[i] / z * v[i, c] for i in range(j + 1))
    return out


def test_attention_brute_force():
    rng = np.random.default_rng(2)
    q, k, v = (rng.normal(size=(6, 5)) for _ in range(3))
    got = oracle.causal_self_attention(q, k, v, 1)
    assert np.max(np.abs(got - _brute_attention(q, k, v))) < 1e-12


def test_attention_single_token_returns_value():
    rng = np.random.default_rng(3)
    q, k, v = (rng.normal(size=(1, 8)) for _ in range(3))
    assert np.array_equal(oracle.causal_self_attention(q, k, v, 2), v)


def test_attention_identical_keys_is_prefix_mean():
    rng = np.random.default_rng(4)
    T = 9
    q = rng.normal(size=(T, 4))
    k = np.tile(rng.normal(size=(1, 4)), (T, 1))
    v = rng.normal(size=(T, 4))
    ref = np.cumsum(v, axis=0) / np.arange(1, T + 1)[:, None]
    assert np.max(np.abs(oracle.causal_self_attention(q, k, v, 1) - ref)) < 1e-12


def test_attention_two_tokens_sigmoid_closed_form():
    rng = np.random.default_rng(5)
    q, k, v = (rng.normal(size=(2, 3)) for _ in range(3))
    p0 = 1.0 / (1.0 + math.exp(-(q[1] @ (k[0] - k[1]))))
    ref1 = p0 * v[0] + (1 - p0) * v[1]
    got = oracle.causal_self_attention(q, k, v, 1)
    assert np.array_equal(got[0], v[0])
    assert np.max(np.abs(got[1] - ref1)) < 1e-14


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(6)
    T, H, hd = 13, 3, 8
    q, k, v = (rng.normal(size=(T, H * hd)) for _ in range(3))

    def heads(a):
        return torch.from_numpy(a).view(T, H, hd).transpose(0, 1)

    ref = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True, scale=1.0)
    ref = ref.transpose(0, 1).reshape(T, H * hd).numpy()
    got = oracle.causal_self_attention(q, k, v, H)
    assert np.max(np.abs(got - ref)) < 1e-12


def test_attention_weights_rows_sum_to_one_and_are_causal():
    rng = np.random.default_rng(7)
    p = oracle.attention_weights(rng.normal(size=(10, 4)), rng.normal(size=(10, 4)))
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-14)
    assert np.all(p[np.triu_indices(10, 1)] == 0.0)


# ----------------------------------------------------------------------------
# LoRA
# ----------------------------------------------------------------------------

def test_lora_delta_equals_merged_weight_and_brute_force():
    rng = np.random.default_rng(8)
    d_in, d_out, r, s = 12, 10, 3, 2.0
    u = rng.normal(size=(5, d_in))
    A = rng.normal(size=(r, d_in))  # stored [r, d_in]
    B = rng.normal(size=(d_out, r))  # stored [d_out, r]
    W = rng.normal(size=(d_out, d_in))
    merged = W + s * (B @ A)  # W' = W + A B in the paper's orientation
    unmerged = u @ W.T + oracle.lora_delta(u, A, B, s)
    assert np.max(np.abs(unmerged - u @ merged.T)) < 1e-12
    brute = np.zeros((5, d_out))
    for m in range(5):
        for n in range(d_out):
            brute[m, n] = s * sum(sum(u[m, i] * A[j, i] for i in range(d_in)) * B[n, j]
                                  for j in range(r))
    assert np.max(np.abs(oracle.lora_delta(u, A, B, s) - brute)) < 1e-12


def test_lora_zero_b_is_bit_identical_to_base():
    w0 = MINI.with_(lora_zero_b=True)
    lz, tz = oracle.prefill_first_token(w0, adapter_of_seq=(0, 1, 1))
    lb, tb = oracle.prefill_first_token(w0, adapter_of_seq=(-1, -1, -1))
    assert np.array_equal(lz, lb) and np.array_equal(tz, tb)
    # a nonzero B does change the result
    ln, _ = oracle.prefill_first_token(MINI, adapter_of_seq=(0, 1, 1))
    assert np.max(np.abs(ln - lb)) > 1e-3


# ----------------------------------------------------------------------------
# causality, embedding and LM head
# ----------------------------------------------------------------------------

def test_causality_later_tokens_do_not_change_earlier_positions():
    toks = synth.tokens(MINI)
    t = 3
    toks2 = toks.copy()
    toks2[:, t + 1:] = (toks2[:, t + 1:] + 11) % (MINI.vocab - 2) + 2
    _, _, h1 = oracle.prefill_first_token(MINI, tokens=toks, keep_hidden=True)
    _, _, h2 = oracle.prefill_first_token(MINI, tokens=toks2, keep_hidden=True)
    T = MINI.seq_len
    for a, b in zip(h1, h2):
        a = a.reshape(MINI.batch, T, -1)
        b = b.reshape(MINI.batch, T, -1)
        assert np.array_equal(a[:, : t + 1], b[:, : t + 1])
        assert not np.array_equal(a[:, t + 1:], b[:, t + 1:])


def test_zero_layers_is_embedding_then_lm_head():
    toks = synth.tokens(MINI)
    logits, tok = oracle.prefill_first_token(MINI, tokens=toks, n_layers=0)
    G = _torch_globals(MINI)
    T = MINI.seq_len
    x = F.embedding(torch.from_numpy(toks[:, -1].astype(np.int64)), G["embed"]) + G["pos"][T - 1]
    ref = F.linear(F.layer_norm(x, (MINI.d_model,), G["lnf_g"], G["lnf_b"], 1e-5), G["embed"])
    assert np.max(np.abs(logits - ref.numpy())) < 1e-12
    assert np.array_equal(tok, np.argmax(ref.numpy().astype(np.float32), axis=1))


def test_greedy_token_takes_lowest_index_on_ties():
    logits = np.array([[0.5, 2.0, 2.0, -1.0], [3.0, 3.0, 3.0, 3.0]])
    assert list(oracle.greedy_token(logits)) == [1, 0]


# ----------------------------------------------------------------------------
# widening of stored values (the weights are the fp16 / bf16 values, widened
# exactly: the model's storage types)
# ----------------------------------------------------------------------------

# bfloat16 is the top half of an IEEE binary32: sign, 8 exponent bits (bias
# 127), 7 fraction bits; binary16 has 5 exponent bits (bias 15), 10 fraction bits
BF16_KNOWN = [
    (0x0000, 0.0), (0x8000, -0.0), (0x3F80, 1.0), (0xBF80, -1.0), (0xC000, -2.0),
    (0x3F81, 1.0 + 2.0 ** -7), (0x4049, 3.140625), (0x3C23, 0.00994873046875),
    (0x0080, 2.0 ** -126),                      # smallest normal
    (0x0001, 2.0 ** -133),                      # smallest subnormal: 2^-126 * 2^-7
    (0x007F, (2.0 ** -7) * 127 * 2.0 ** -126),  # largest subnormal
    (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127),   # largest finite
    (0x7F80, math.inf), (0xFF80, -math.inf),
]
F16_KNOWN = [
    (0x0000, 0.0), (0x3C00, 1.0), (0xC000, -2.0), (0x3C01, 1.0 + 2.0 ** -10),
    (0x0001, 2.0 ** -24), (0x0400, 2.0 ** -14), (0x7BFF, 65504.0), (0x7C00, math.inf),
    (0xFC00, -math.inf),
]


@pytest.mark.parametrize("kind,table", [("bf16", BF16_KNOWN), ("f16", F16_KNOWN)])
def test_widen_known_bit_patterns(kind, table):
    bits = np.array([b for b, _ in table], dtype=np.uint16)
    got = oracle.widen(bits, kind)
    for (b, v), g in zip(table, got):
        assert g == v and math.copysign(1.0, g) == math.copysign(1.0, v), (hex(b), g, v)
    nan = oracle.widen(np.array([0x7FC0, 0xFFC1, 0x7F81], np.uint16), "bf16")
    assert np.all(np.isnan(nan))


def test_widen_bf16_matches_torch_on_every_pattern():
    # all 65536 words: torch's bfloat16 -> float64 conversion is an independent
    # implementation of the same definition
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(bits, "bf16")
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert np.all(same)
    assert np.array_equal(np.signbit(got), np.signbit(ref))


def test_widen_f16_matches_numpy_on_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(bits, "f16")
    ref = bits.view(np.float16).astype(np.float64)
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert np.all(same)


def test_widen_bf16_is_exact_for_rounded_draws():
    # a bf16 storage draw widened must equal the float32 draw rounded to bf16
    f32 = synth.normal(21, 5, (20_000,), 0.0, 0.02, "f32")
    bf = synth.normal(21, 5, (20_000,), 0.0, 0.02, "bf16")
    ref = torch.from_numpy(f32).to(torch.bfloat16).double().numpy()
    assert np.array_equal(oracle.widen(bf, "bf16"), ref)
    # rounding moves a value by at most half a unit in the last of 8 bits
    assert np.all(np.abs(oracle.widen(bf, "bf16") - f32) <= np.abs(f32) * 2.0 ** -8)


# ----------------------------------------------------------------------------
# independent float64 build from library routines
# ----------------------------------------------------------------------------

def _t_widen(a, kind):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if kind == "f32":
        return t.double()
    if kind == "f16":
        return t.view(torch.float16).double()
    return t.view(torch.bfloat16).double()


def _kind(w):
    return "f32" if w.oracle_weights == "f32" else w.dtype


def _torch_globals(w):
    k = _kind(w)
    return {n: _t_widen(synth.base_tensor(w, -1, n, k), k) for n in synth.GLOBAL_TENSORS}


def torch_prefill(w, toks, adapters):
    """Whole prefill from torch.nn.functional routines, LoRA merged per sequence."""
    k = _kind(w)
    G = _torch_globals(w)
    B, T = toks.shape
    d, H = w.d_model, w.n_heads
    x = F.embedding(torch.from_numpy(toks.astype(np.int64)), G["embed"]) + G["pos"][:T]
    s = w.lora_scale
    for layer in range(w.n_layers):
        W = {n: _t_widen(synth.base_tensor(w, layer, n, k), k) for n in synth.LAYER_TENSORS}
        out = []
        for b in range(B):
            Wb = dict(W)
            a = adapters[b]
            if a >= 0:
                for t in w.lora_targets:
                    A = _t_widen(synth.lora_tensor(w, a, layer, t, "A", k), k)
                    Bm = _t_widen(synth.lora_tensor(w, a, layer, t, "B", k), k)
                    Wb["w" + t] = W["w" + t] + s * (Bm @ A)  # merged weight
            xb = x[b]
            u = F.layer_norm(xb, (d,), Wb["ln1_g"], Wb["ln1_b"], w.ln_eps)
            q = F.linear(u, Wb["wq"], Wb["bq"]).view(T, H, -1).transpose(0, 1)
            kk = F.linear(u, Wb["wk"], Wb["bk"]).view(T, H, -1).transpose(0, 1)
            v = F.linear(u, Wb["wv"], Wb["bv"]).view(T, H, -1).transpose(0, 1)
            o = F.scaled_dot_product_attention(q, kk, v, is_causal=True)  # default 1/sqrt(hd)
            o = o.transpose(0, 1).reshape(T, d)
            xb = xb + F.linear(o, Wb["wo"], Wb["bo"])
            hb = F.relu(F.linear(F.layer_norm(xb, (d,), Wb["ln2_g"], Wb["ln2_b"], w.ln_eps),
                                 Wb["w1"], Wb["b1"]))
            out.append(xb + F.linear(hb, Wb["w2"], Wb["b2"]))
        x = torch.stack(out)
    z = F.layer_norm(x[:, -1], (d,), G["lnf_g"], G["lnf_b"], w.ln_eps)
    return F.linear(z, G["embed"]).numpy()


@pytest.mark.parametrize("name", ["mini", "mini-bf16", "tiny"])
def test_oracle_matches_independent_library_build(name):
    w = {"mini": MINI, "mini-bf16": MINI_BF16, "tiny": TINY}[name]
    toks = synth.tokens(w)
    ad = w.adapters()
    logits, tok = oracle.prefill_first_token(w, tokens=toks)
    ref = torch_prefill(w, toks, ad)
    scale = np.max(np.abs(ref))
    assert np.max(np.abs(logits - ref)) < 1e-11 * max(1.0, scale)
    assert np.array_equal(tok, np.argmax(ref.astype(np.float32), axis=1))


# ----------------------------------------------------------------------------
# planted mistakes must be caught
# ----------------------------------------------------------------------------

def _ln_unbiased(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(x.var(axis=-1, ddof=1, keepdims=True) + eps) * g + b


def _ln_no_beta(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(((x - mu) ** 2).mean(axis=-1, keepdims=True) + eps) * g


def _attn_not_causal(q, k):
    s = q @ k.T
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    return p / p.sum(axis=1, keepdims=True)


def _attn_off_by_one(q, k):
    T = q.shape[0]
    s = q @ k.T
    allowed = np.tril(np.ones((T, T), dtype=bool), -1)
    allowed[0, 0] = True
    s = np.where(allowed, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    p = np.where(allowed, np.exp(s), 0.0)
    return p / p.sum(axis=1, keepdims=True)


def _lora_wrong_sign(u, A, B, scale):
    return -scale * ((u @ A.T) @ B.T)


def _lora_wrong_scale(u, A, B, scale):
    return ((u @ A.T) @ B.T) / scale


MUTANTS = {
    "layer_norm": [_ln_unbiased, _ln_no_beta],
    "attention_weights": [_attn_not_causal, _attn_off_by_one],
    "lora_delta": [_lora_wrong_sign, _lora_wrong_scale],
}


@pytest.mark.parametrize("fname,idx", [(f, i) for f, ms in MUTANTS.items() for i in range(len(ms))])
def test_planted_mistakes_are_caught(monkeypatch, fname, idx):
    toks = synth.tokens(MINI)
    ref = torch_prefill(MINI, toks, MINI.adapters())
    monkeypatch.setattr(ol, fname, MUTANTS[fname][idx])
    logits, _ = ol.prefill_first_token(MINI, tokens=toks)
    assert np.max(np.abs(logits - ref)) > 1e-6


def _widen_bf16_shifted(a, kind):
    # a plausible slip: the bfloat16 word shifted into the wrong half
    if kind == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
        return bits.view(np.float32).astype(np.float64)
    return _WIDEN(a, kind)


_WIDEN = ol.widen


def test_planted_widening_mistake_is_caught(monkeypatch):
    toks = synth.tokens(MINI_BF16)
    ref = torch_prefill(MINI_BF16, toks, MINI_BF16.adapters())
    monkeypatch.setattr(ol, "widen", _widen_bf16_shifted)
    monkeypatch.setattr(oracle, "widen", _widen_bf16_shifted)
    logits, _ = ol.prefill_first_token(MINI_BF16, tokens=toks)
    assert not np.all(np.isfinite(logits)) or np.max(np.abs(logits - ref)) > 1e-6
    with pytest.raises(AssertionError):
        test_widen_known_bit_patterns("bf16", BF16_KNOWN)
