"""Plain, slow, float64 oracle of the OPT-style prefill with unmerged LoRA.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import or run this module.  It shares
no code with the GPU path; its only input dependency is the seeded generator
in ``synth`` (weights and tokens), which holds none of this arithmetic.

What it computes (PipeBoost, arXiv 2503.17707):

* Prefill (Section 2.1, "LLM Serving"): the prompt tokens enter the first
  layer; every layer applies self-attention across the prompt tokens and then
  a feed-forward network, its output feeds the next layer, and the last layer
  produces the first output token.  The models are OPT-family decoders
  (Section 5, which adapts OPT, Falcon and Mistral): learned absolute position
  embeddings, pre-LayerNorm blocks, ReLU FFN, final LayerNorm, LM head tied to
  the token embedding.
* LoRA (Section 2.1): the base weight W stays fixed and a low-rank pair A
  (d x r) and B (r x d) adds its product.  Section 4.3.2 merges the pair into
  W before inference; the unmerged form computed here gives the same result in
  exact arithmetic, and different sequences of one batch may use different
  adapters on the shared base.
* The paper's contribution (Sections 4.2 and 4.3) is when each layer may
  start, not what it computes, so the layer load order never appears here.

Readings where the paper is silent (listed with the design notes): no
position offset; biases on q, k, v, o, fc1, fc2; LoRA scale alpha/r; q is
divided by sqrt(head_dim) after its bias and LoRA delta; LayerNorm uses the
biased variance and eps = 1e-5; masked attention positions are excluded;
greedy decoding takes the lowest index among equal maxima, decided on float32
logits (the precision the GPU computes them in).

Storage layout of the inputs (from ``synth``): every matrix is [out, in];
LoRA A is stored [r, d_in] (the paper's A transposed) and B [d_out, r] (the
paper's B transposed).

All arithmetic is float64.
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Sequence

import numpy as np

import synth


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def widen(a: np.ndarray, kind: str) -> np.ndarray:
    """Exact widening of stored values to float64.

    ``kind`` is the storage type: "f32" (float32 values), "f16" (IEEE binary16
    bit patterns) or "bf16" (bfloat16 bit patterns, the top half of a float32).
    """
    if kind == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if kind == "f16":
        return np.asarray(a, dtype=np.uint16).view(np.float16).astype(np.float64)
    if kind == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(kind)


class WeightSource:
    """Draws a workload's tensors from ``synth`` and widens them to float64.

    For a workload whose ``oracle_weights`` is "f32" the oracle uses the float
    draws themselves (the GPU stores their rounding to its dtype); otherwise the
    stored fp16/bf16 values are the model.
    """

    def __init__(self, w: synth.Workload):
        self.w = w
        self.kind = "f32" if w.oracle_weights == "f32" else w.dtype

    def globals(self) -> Dict[str, np.ndarray]:
        return {n: widen(synth.base_tensor(self.w, -1, n, self.kind), self.kind)
                for n in synth.GLOBAL_TENSORS}

    def layer(self, layer: int) -> Dict[str, np.ndarray]:
        return {n: widen(synth.base_tensor(self.w, layer, n, self.kind), self.kind)
                for n in synth.LAYER_TENSORS}

    def lora(self, adapter: int, layer: int) -> Dict[str, Dict[str, np.ndarray]]:
        out = {}
        for t in self.w.lora_targets:
            out[t] = {x: widen(synth.lora_tensor(self.w, adapter, layer, t, x, self.kind), self.kind)
                      for x in ("A", "B")}
        return out


# ----------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------

def layer_norm(x: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis (the pre-LN blocks of the OPT family, Section 5).

    (v - mean(v)) / sqrt(var(v) + eps) * gamma + beta, with the biased variance.
    """
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gamma + beta


def lora_delta(u: np.ndarray, A: np.ndarray, B: np.ndarray, scale: float) -> np.ndarray:
    """Unmerged LoRA delta, Section 2.1: scale * u A B in the paper's notation.

    A is stored [r, d_in] and B [d_out, r], so the product is scale * (u A^T) B^T.
    """
    return scale * ((u @ A.T) @ B.T)


def attention_weights(q: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Causal softmax weights of one head (Section 2.1, self-attention in prefill).

    Row j holds softmax over positions 0..j of q_j . k_i; positions after j are
    excluded (weight exactly 0).  q is already divided by sqrt(head_dim).
    """
    T = q.shape[0]
    s = q @ k.T
    allowed = np.tril(np.ones((T, T), dtype=bool))
    s = np.where(allowed, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    p = np.where(allowed, np.exp(s), 0.0)
    return p / p.sum(axis=1, keepdims=True)


def causal_self_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Multi-head causal self-attention of one sequence; q, k, v are [T, d].

    Heads are consecutive slices of head_dim columns; the output concatenates
    the heads back into [T, d].
    """
    T, d = q.shape
    hd = d // n_heads
    out = np.empty((T, d), dtype=np.float64)
    for h in range(n_heads):
        sl = slice(h * hd, (h + 1) * hd)
        p = attention_weights(q[:, sl], k[:, sl])
        out[:, sl] = p @ v[:, sl]
    return out


def decoder_layer(x: np.ndarray, W: Dict[str, np.ndarray], n_heads: int, eps: float,
                  seq_len: int, lora_of_seq: Sequence[Optional[Dict[str, Dict[str, np.ndarray]]]],
                  scale: float) -> np.ndarray:
    """One pre-LN OPT decoder block over a batch of sequences.

    x is the residual stream [B*T, d] (sequence-major).  lora_of_seq[b] maps a
    target ("q", "k", "v", "o") to its {"A", "B"} pair for sequence b, or is
    None for the base model.
    """
    n, d = x.shape
    hd = d // n_heads
    u = layer_norm(x, W["ln1_g"], W["ln1_b"], eps)
    proj = {"q": (W["wq"], W["bq"]), "k": (W["wk"], W["bk"]), "v": (W["wv"], W["bv"])}
    qkv = {}
    for t, (wt, bt) in proj.items():
        y = u @ wt.T + bt
        for b, lo in enumerate(lora_of_seq):
            if lo is not None and t in lo:
                rows = slice(b * seq_len, (b + 1) * seq_len)
                y[rows] += lora_delta(u[rows], lo[t]["A"], lo[t]["B"], scale)
        qkv[t] = y
    q = qkv["q"] / np.sqrt(hd)
    attn = np.empty_like(x)
    for b in range(len(lora_of_seq)):
        rows = slice(b * seq_len, (b + 1) * seq_len)
        attn[rows] = causal_self_attention(q[rows], qkv["k"][rows], qkv["v"][rows], n_heads)
    y = attn @ W["wo"].T + W["bo"]
    for b, lo in enumerate(lora_of_seq):
        if lo is not None and "o" in lo:
            rows = slice(b * seq_len, (b + 1) * seq_len)
            y[rows] += lora_delta(attn[rows], lo["o"]["A"], lo["o"]["B"], scale)
    x = x + y
    h = layer_norm(x, W["ln2_g"], W["ln2_b"], eps) @ W["w1"].T + W["b1"]
    h = np.maximum(h, 0.0)
    return x + (h @ W["w2"].T + W["b2"])


def final_logits(x_last: np.ndarray, G: Dict[str, np.ndarray], eps: float) -> np.ndarray:
    """Final LayerNorm of each sequence's last position, then the tied LM head."""
    z = layer_norm(x_last, G["lnf_g"], G["lnf_b"], eps)
    return z @ G["embed"].T


def greedy_token(logits: np.ndarray) -> np.ndarray:
    """Greedy first token: the lowest index among the maxima of float32 logits."""
    return np.argmax(np.asarray(logits, dtype=np.float32), axis=-1).astype(np.int32)


# ----------------------------------------------------------------------------
# whole prefill
# ----------------------------------------------------------------------------

def prefill_first_token(w: synth.Workload, tokens: Optional[np.ndarray] = None,
                        adapter_of_seq: Optional[Iterable[int]] = None,
                        source: Optional[WeightSource] = None,
                        n_layers: Optional[int] = None,
                        keep_hidden: bool = False):
    """Prefill of a batch of equal-length prompts, returning the first token.

    Returns (logits [B, V] float64, tokens [B] int32) and, with keep_hidden,
    the residual stream after each layer as a third element.  n_layers runs
    only the first layers (used to time a bounded sample).
    """
    src = source or WeightSource(w)
    toks = synth.tokens(w) if tokens is None else np.asarray(tokens, dtype=np.int64)
    B, T = toks.shape
    adapters = list(w.adapters() if adapter_of_seq is None else adapter_of_seq)
    G = src.globals()
    # embedding: token row plus the learned position row of the same index
    x = G["embed"][toks.reshape(-1)] + np.tile(G["pos"][:T], (B, 1))
    hidden: List[np.ndarray] = []
    L = w.n_layers if n_layers is None else n_layers
    for layer in range(L):
        W = src.layer(layer)
        cache = {}
        lora_of_seq = []
        for a in adapters:
            if a < 0:
                lora_of_seq.append(None)
                continue
            if a not in cache:
                cache[a] = src.lora(a, layer)
            lora_of_seq.append(cache[a])
        x = decoder_layer(x, W, w.n_heads, w.ln_eps, T, lora_of_seq, w.lora_scale)
        if keep_hidden:
            hidden.append(x.copy())
    x_last = x.reshape(B, T, -1)[:, T - 1, :]
    logits = final_logits(x_last, G, w.ln_eps)
    tok = greedy_token(logits)
    if keep_hidden:
        return logits, tok, hidden
    return logits, tok
