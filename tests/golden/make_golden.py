"""Write the oracle's first-token logits for the full-size workloads.

Calls only the CPU oracle (and the shared seeded generator for its inputs):
    python tests/golden/make_golden.py opt-1.3b opt-6.7b opt-13b opt-66b
    python tests/golden/make_golden.py --decode 2 opt-1.3b

Each workload gives tests/golden/<name>.npz with
  logits  float32 [B, V]  last-position logits (oracle float64, rounded once)
  tokens  int32   [B]     greedy first tokens
  margin  float64 [B]     top-1 minus top-2 logit (how far from a tie)
  meta    str             JSON: workload fields and oracle wall time
With --decode K it writes tests/golden/<name>-decode.npz instead: the same
fields stacked over K greedy steps after the first token ([K, B, V], [K, B],
[K, B]), step k being the oracle prefill of the prompt plus the oracle's own
first k tokens.
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


def make_decode(name: str, steps: int) -> str:
    w = synth.WORKLOADS[name]
    t0 = time.time()
    seq = synth.tokens(w).astype(np.int64)
    _, tok = oracle.prefill_first_token(w, tokens=seq)
    out_logits, out_tok, out_margin = [], [], []
    for _ in range(steps):
        seq = np.concatenate([seq, tok[:, None].astype(np.int64)], axis=1)
        logits, tok = oracle.prefill_first_token(w, tokens=seq)
        srt = np.sort(logits, axis=1)
        out_logits.append(logits.astype(np.float32))
        out_tok.append(tok.astype(np.int32))
        out_margin.append(srt[:, -1] - srt[:, -2])
    dt = time.time() - t0
    meta = {"workload": dataclasses.asdict(w), "oracle_seconds": dt, "dtype": "float64",
            "decode_steps": steps}
    out = os.path.join(HERE, name + "-decode.npz")
    np.savez_compressed(out, logits=np.stack(out_logits), tokens=np.stack(out_tok),
                        margin=np.stack(out_margin), meta=np.array(json.dumps(meta)))
    print("%s decode: %.1f s, tokens %s" % (name, dt, np.stack(out_tok).tolist()), flush=True)
    return out


if __name__ == "__main__":
    args = sys.argv[1:]
    if args[:1] == ["--decode"]:
        k = int(args[1])
        for n in args[2:] or ["opt-1.3b"]:
            make_decode(n, k)
    else:
        for n in args or ["opt-1.3b", "opt-6.7b", "opt-13b", "opt-66b"]:
            make(n)
