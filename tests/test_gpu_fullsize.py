"""Full-size OPT-shaped workloads on the HIP path, against the oracle's stored
first-token logits (tests/golden/<name>.npz, written by make_golden.py from
the CPU oracle alone), plus load-order bit-identity at full size."""
import os
import time

import numpy as np
import pytest

import synth
from gpu_common import compare, golden_path, log

pytestmark = pytest.mark.gpu


def _golden(name):
    p = golden_path(name)
    if not os.path.exists(p):
        pytest.skip("oracle logits for %s not generated" % name)
    g = np.load(p, allow_pickle=False)
    return g["logits"], g["tokens"]


def _cold_start(name, orders):
    from paper_2503_17707_amd import binding as pb

    w = synth.WORKLOADS[name]
    t0 = time.time()
    log("case", name, "generating pinned host weights")
    hw, m = pb.setup(w)
    log("  weights ready in %.1f s" % (time.time() - t0))
    outs = []
    try:
        toks = synth.tokens(w)
        for o in orders:
            m.poison(0xFF)
            pb.attach_all(m, hw)
            m.stream_layers(hw, o)
            tok, logits = m.prefill(toks, w.adapters())
            b, ms = m.load_stats()
            log("  order %s..: load %.1f ms (%.1f GB/s), tokens %s" % (
                list(o)[:4], ms, b / ms / 1e6, list(tok)))
            outs.append((tok, logits))
    finally:
        m.destroy()
        hw.free()
    return outs


@pytest.mark.parametrize("name", ["opt-1.3b", "opt-6.7b"])
def test_fullsize_matches_oracle(name):
    ref_logits, ref_tok = _golden(name)
    w = synth.WORKLOADS[name]
    (tok, logits), = _cold_start(name, [w.order()])
    compare(name, logits, tok, ref_logits, ref_tok)


def test_opt13b_rotated_order_matches_oracle_and_natural_order_bitwise():
    name = "opt-13b"
    ref_logits, ref_tok = _golden(name)
    w = synth.WORKLOADS[name]
    outs = _cold_start(name, [w.order(), list(range(w.n_layers))])
    compare(name, outs[0][1], outs[0][0], ref_logits, ref_tok)
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1].view(np.uint32), outs[1][1].view(np.uint32))


def test_opt66b_matches_oracle():
    name = "opt-66b"
    ref_logits, ref_tok = _golden(name)
    w = synth.WORKLOADS[name]
    (tok, logits), = _cold_start(name, [w.order()])
    compare(name, logits, tok, ref_logits, ref_tok)
