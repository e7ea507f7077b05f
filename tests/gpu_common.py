"""Helpers of the GPU tests: run the HIP path through the C ABI and compare."""
import os
import sys

import numpy as np

import synth

# parity bar for first-token logits (fp32 on the GPU vs the float64 oracle)
MAX_ABS = 3e-2
MAX_REL_L2 = 1e-2


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare(tag, got_logits, got_tok, ref_logits, ref_tok, max_abs=MAX_ABS):
    ref = np.asarray(ref_logits, dtype=np.float64)
    got = np.asarray(got_logits, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s: non-finite logits" % tag
    d = np.abs(got - ref)
    maxd = float(d.max())
    # relative L2 of each sequence's logits; the bar holds for the worst one
    rows = np.linalg.norm(got - ref, axis=-1) / np.linalg.norm(ref, axis=-1)
    rel = float(np.max(rows))
    srt = np.sort(ref, axis=1)
    margin = srt[:, -1] - srt[:, -2]
    log("%s: max|d|=%.3e rel_l2 per sequence=%s tokens gpu=%s oracle=%s margin=%s" % (
        tag, maxd, np.array2string(rows, precision=3), list(got_tok), list(ref_tok),
        np.round(margin, 4).tolist()))
    assert maxd <= max_abs, "%s: max|d| %.3e > %.3e" % (tag, maxd, max_abs)
    assert rel <= MAX_REL_L2, "%s: rel L2 %.3e > %.1e" % (tag, rel, MAX_REL_L2)
    assert list(got_tok) == list(ref_tok), "%s: greedy tokens differ (margins %s)" % (tag, margin)
    return maxd, rel


def run_gpu(w, order=None, hw=None, adapters=None, tokens=None, free=True, **cap):
    """Full cold start through the C ABI: attach adapters, stream layers, prefill."""
    from paper_2503_17707_amd import binding as pb

    hw_, m = pb.setup(w, hw=hw, **cap)
    try:
        pb.attach_all(m, hw_)
        m.stream_layers(hw_, order if order is not None else w.order())
        toks = synth.tokens(w) if tokens is None else tokens
        ad = list(w.adapters() if adapters is None else adapters)
        tok, logits = m.prefill(toks, ad)
        return tok, logits
    finally:
        m.destroy()
        if free and hw is None:
            hw_.free()


def golden_path(name):
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", name + ".npz")
