"""Float32 CPU build of the decoder that rounds activations to the storage dtype.

Test infrastructure, not a reference of the kernels' arithmetic: it models
only the precision of activation storage. Activations are rounded to bf16 or
fp16 wherever the GPU path stores them in the weights' dtype:
- the LayerNorm outputs;
- the LoRA shrink outputs;
- q (after its 1/sqrt(head_dim) scale), k and v;
- the attention probabilities, which are the operand of the P V product
  and whose rounded values make up the row sum;
- the attention output;
- the FFN hidden layer after ReLU.

Everything else is float32: the residual stream, the products' accumulation,
the final LayerNorm and the logits. The gap between its logits and those of
the float64 oracle is therefore the error that storing activations in that
dtype brings by itself, whatever the kernels. The decoder follows Section 2.1
(pre-LayerNorm OPT layers, unmerged LoRA y = xW + s (xA) B).

The GPU path rounds a few intermediates that this model does not, and the
model rounds none of the GPU path's other steps. So it gives the size of the
storage error, not the GPU path's exact values. Weights are the stored words,
widened exactly, as the oracle's storage mode reads them.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

import synth


def _widen(a, kind):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if kind == "f32":
        return t.float()
    return (t.view(torch.float16) if kind == "f16" else t.view(torch.bfloat16)).float()


def _rounder(round_to):
    if round_to is None:
        return lambda t: t
    dt = {"bf16": torch.bfloat16, "f16": torch.float16}[round_to]
    return lambda t: t.to(dt).float()


def storage_rounded_logits(w, round_to):
    """Last-position logits [B, V] (float64 array) of workload `w`, activations
    rounded to `round_to` ("bf16", "f16", or None for no rounding)."""
    k = "f32" if w.oracle_weights == "f32" else w.dtype
    r = _rounder(round_to)
    G = {n: _widen(synth.base_tensor(w, -1, n, k), k) for n in synth.GLOBAL_TENSORS}
    toks = synth.tokens(w)
    ad = w.adapters()
    B, T = toks.shape
    d, H = w.d_model, w.n_heads
    hd = d // H
    s = w.lora_scale
    causal = torch.triu(torch.full((T, T), float("-inf")), 1)
    x = F.embedding(torch.from_numpy(toks.astype(np.int64)), G["embed"]) + G["pos"][:T]
    for layer in range(w.n_layers):
        W = {n: _widen(synth.base_tensor(w, layer, n, k), k) for n in synth.LAYER_TENSORS}
        out = []
        for b in range(B):
            lora = {}
            if ad[b] >= 0:
                for t in w.lora_targets:
                    lora[t] = (_widen(synth.lora_tensor(w, ad[b], layer, t, "A", k), k),
                               _widen(synth.lora_tensor(w, ad[b], layer, t, "B", k), k))

            def proj(inp, t):
                y = inp @ W["w" + t].T + W["b" + t]
                if t in lora:
                    A, Bm = lora[t]
                    y = y + s * (r(inp @ A.T) @ Bm.T)
                return y

            xb = x[b]
            u = r(F.layer_norm(xb, (d,), W["ln1_g"], W["ln1_b"], w.ln_eps))
            q = r(proj(u, "q") / math.sqrt(hd)).view(T, H, hd).transpose(0, 1)
            kk = r(proj(u, "k")).view(T, H, hd).transpose(0, 1)
            v = r(proj(u, "v")).view(T, H, hd).transpose(0, 1)
            S = q @ kk.transpose(1, 2) + causal
            P = r(torch.exp(S - S.max(dim=-1, keepdim=True).values))
            o = r(((P @ v) / P.sum(dim=-1, keepdim=True)).transpose(0, 1).reshape(T, d))
            xb = xb + proj(o, "o")
            h = r(F.layer_norm(xb, (d,), W["ln2_g"], W["ln2_b"], w.ln_eps))
            f = r(F.relu(h @ W["w1"].T + W["b1"]))
            out.append(xb + f @ W["w2"].T + W["b2"])
        x = torch.stack(out)
    z = F.layer_norm(x[:, -1], (d,), G["lnf_g"], G["lnf_b"], w.ln_eps)
    return (z @ G["embed"].T).double().numpy()
