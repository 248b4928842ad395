"""Writes many_rows_8b_golden.json: the oracle's ready distribution for a 300-token entry
on the 8B-shaped decoder (32 layers, 1024 synthetic persistent cells, uniform token ids):
its top logits, 256 sampled logits, argmax, gap and log-sum-exp.  More than 256 entry rows
put every projection on the library's 64-row-tile plans (those of the batched pass), so
this pins that path over the full depth.  Calls only the oracle and the seeded input
generator.

    python tests/golden/make_many_rows_golden.py     (a few minutes on 8 cores)
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

SEED, N_PAST, M, STREAM = 1002, 1024, 300, 77


def main():
    shape = synth.M8B
    entry = synth.cpu_tokens(M, SEED, STREAM, shape.vocab)
    t0 = time.time()
    w = oracle.Weights(shape, SEED, cache_layers=False)
    kv = oracle.KVState(shape, N_PAST + M, seed=SEED, n_synth=N_PAST)
    logits = oracle.forward(w, kv, N_PAST, entry, drop_layers=True, last_only=True)
    s = oracle.summary(logits)
    order = np.argsort(-logits, kind="stable")[:32]
    sample_idx = np.unique(synth.cpu_tokens(256, SEED, 98, shape.vocab))
    out = {
        "shape": "8b", "seed": SEED, "n_past": N_PAST, "entry_stream": STREAM, "m": M,
        "argmax": s.argmax, "second": s.second, "top1": s.top1, "top2": s.top2, "gap": s.gap,
        "lse": s.lse,
        "top_idx": [int(i) for i in order], "top_val": [float(logits[i]) for i in order],
        "sample_idx": [int(i) for i in sample_idx],
        "sample_val": [float(logits[i]) for i in sample_idx],
        "seconds": time.time() - t0,
    }
    with open(os.path.join(HERE, "many_rows_8b_golden.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(f"argmax {s.argmax} gap {s.gap:.4f} lse {s.lse:.4f} in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
