"""Writes <workload>_golden.json for the full-depth workloads named on the command line
(default: target32b agentic8b): the oracle's ready distribution for the workload's first
entry over every layer, with its synthetic persistent cells and its LM-head bias if it has
one -- the top logits, 256 sampled logits, argmax, gap and log-sum-exp.  Calls only the
oracle and the seeded input generator.

  target32b: 64 layers, d 5120, 64/8 heads x 128, SwiGLU 27648, vocab 152064; 16384
             cells, a 32-token entry, bias 10.1 on the planted fast-answer token
  agentic8b: 32 layers, d 4096, 32/8 heads x 128, SwiGLU 14336, vocab 128256; 32768
             cells, a 128-token envelope
  stream70b_mxfp4: 80 layers, d 8192, 64/8 heads x 128, SwiGLU 28672, vocab 128256,
             MXFP4 projections; 8192 cells, a 32-token entry (about 40 minutes)

    python tests/golden/make_full_depth_golden.py [workload ...]   (minutes on 8 cores)
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


def write(name: str) -> None:
    wl = synth.WORKLOADS[name]
    entry = synth.entry_tokens(wl, 0)
    bias = synth.workload_bias(wl)
    t0 = time.time()
    w = oracle.Weights(wl.shape, wl.seed, lm_bias=bias, cache_layers=False)
    kv = oracle.KVState(wl.shape, wl.n_past + len(entry), seed=wl.seed, n_synth=wl.n_past)
    logits = oracle.forward(w, kv, wl.n_past, entry, drop_layers=True, last_only=True)
    s = oracle.summary(logits)
    order = np.argsort(-logits, kind="stable")[:32]
    sample_idx = np.unique(synth.cpu_tokens(256, wl.seed, 99, wl.shape.vocab))
    out = {
        "workload": name, "seed": wl.seed, "n_past": wl.n_past,
        "entry": [int(t) for t in entry], "lm_bias": wl.lm_bias,
        "planted": int(synth.planted_token(wl)),
        "argmax": s.argmax, "second": s.second, "top1": s.top1, "top2": s.top2, "gap": s.gap,
        "lse": s.lse,
        "top_idx": [int(i) for i in order], "top_val": [float(logits[i]) for i in order],
        "sample_idx": [int(i) for i in sample_idx],
        "sample_val": [float(logits[i]) for i in sample_idx],
        "seconds": time.time() - t0,
    }
    with open(os.path.join(HERE, f"{name}_golden.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(f"{name}: argmax {s.argmax} gap {s.gap:.4f} lse {s.lse:.4f} in {time.time() - t0:.0f} s",
          flush=True)


def main():
    for name in sys.argv[1:] or ["target32b", "agentic8b"]:
        write(name)


if __name__ == "__main__":
    main()
