"""Writes stream8b_golden.json: the oracle's ready distribution for the full streaming
workload (8B-shaped decoder, 32 layers, 8192 synthetic persistent cells, a 24-token
query prefix plus an 8-token assistant header) -- its top logits, 256 sampled logits,
argmax, gap and log-sum-exp.  Calls only the oracle and the seeded input generator.

    python tests/golden/make_stream8b_golden.py     (about 5 minutes on 8 cores)
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402


def main():
    wl = synth.WORKLOADS["stream8b"]
    entry = synth.entry_tokens(wl, 0)
    t0 = time.time()
    w = oracle.Weights(wl.shape, wl.seed, cache_layers=False)
    kv = oracle.KVState(wl.shape, wl.n_past + len(entry), seed=wl.seed, n_synth=wl.n_past)
    logits = oracle.forward(w, kv, wl.n_past, entry, drop_layers=True, last_only=True)
    s = oracle.summary(logits)
    order = np.argsort(-logits, kind="stable")[:32]
    sample_idx = np.unique(synth.cpu_tokens(256, wl.seed, 99, wl.shape.vocab))
    out = {
        "workload": "stream8b", "seed": wl.seed, "n_past": wl.n_past,
        "entry": [int(t) for t in entry],
        "argmax": s.argmax, "second": s.second, "top1": s.top1, "top2": s.top2, "gap": s.gap,
        "lse": s.lse,
        "top_idx": [int(i) for i in order], "top_val": [float(logits[i]) for i in order],
        "sample_idx": [int(i) for i in sample_idx],
        "sample_val": [float(logits[i]) for i in sample_idx],
        "seconds": time.time() - t0,
    }
    with open(os.path.join(HERE, "stream8b_golden.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(f"argmax {s.argmax} gap {s.gap:.4f} lse {s.lse:.4f} in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
