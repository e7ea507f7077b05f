"""Write the oracle's first-token logits for the full-size workloads.

Calls only the CPU oracle (and the shared seeded generator for its inputs):
    python tests/golden/make_golden.py opt-1.3b opt-6.7b opt-13b opt-66b

Each workload gives tests/golden/<name>.npz with
  logits  float32 [B, V]  last-position logits (oracle float64, rounded once)
  tokens  int32   [B]     greedy first tokens
  margin  float64 [B]     top-1 minus top-2 logit (how far from a tie)
  meta    str             JSON: workload fields and oracle wall time
"""
import dataclasses
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402


def make(name: str) -> str:
    w = synth.WORKLOADS[name]
    t0 = time.time()
    logits, tok = oracle.prefill_first_token(w)
    dt = time.time() - t0
    srt = np.sort(logits, axis=1)
    margin = srt[:, -1] - srt[:, -2]
    meta = {"workload": dataclasses.asdict(w), "oracle_seconds": dt, "dtype": "float64"}
    out = os.path.join(HERE, name + ".npz")
    np.savez_compressed(out, logits=logits.astype(np.float32), tokens=tok.astype(np.int32),
                        margin=margin, meta=np.array(json.dumps(meta)))
    print("%s: %.1f s, tokens %s, margins %s" % (name, dt, tok.tolist(), np.round(margin, 4).tolist()),
          flush=True)
    return out


if __name__ == "__main__":
    for n in sys.argv[1:] or ["opt-1.3b", "opt-6.7b", "opt-13b", "opt-66b"]:
        make(n)
