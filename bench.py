#!/usr/bin/env python3
"""Benchmark of the speculative pre-positioning hot path on one MI355X.

Workload (the streaming-session configuration): an 8B-shaped decoder (32 layers,
d_model 4096, 32 query / 8 kv heads of dim 128, SwiGLU 14336, vocab 128256) in
bf16 with seeded random weights, a persistent KV cache of n_s = 8192 synthetic
cells, and an entry of 24 query-prefix tokens plus an 8-token assistant header.

One step is the whole hot path: the pre-position (budget check, entry forward pass
over the resident cells with the in-place KV append, LM head with the fused
vocabulary reductions, ready record), the gate scan of the cached distribution
(tau = 2, a 64-token fast-answer set), and the invalidation of the record.
The cells are rewritten at the same positions each step (idempotent).

Prints one JSON line.  `value` is entry tokens per second over the timed steps.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "pre-position step ms & entry tok/s; gate scan µs; % of HBM roofline"
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_gate_up_stream8b_traffic.json")
GEMM_SRC = os.path.join(ROOT, "paper_2606_29565_amd", "csrc", "gemm.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=32,
                    help="decoder layers in the oracle's timed sample")
    ap.add_argument("--no-mxfp4-70b", action="store_true",
                    help="skip the secondary measurement on the 70B-shaped MXFP4 model")
    ap.add_argument("--no-energy", action="store_true",
                    help="skip the energy measurements (seconds of back-to-back pre-positions)")
    ap.add_argument("--mxfp4-70b-only", action="store_true",
                    help="run only the 70B-shaped MXFP4 measurement and print its JSON")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run the library's plain copy kernel 4 times over MIB MiB (the "
                         "known-size reference for scaling the HBM byte counters), then exit")
    return ap.parse_args()


def algorithmic_bytes(shape, M: int, n_past: int) -> dict:
    """Bytes a pre-position step must move at least: every weight once, the KV cells
    read once, the new cells written, activations in and out of each projection.
    MXFP4 projections weigh half a byte per weight plus one scale byte per 32."""
    d, F, V, L = shape.d_model, shape.ffn, shape.vocab, shape.n_layers
    nq, nkv = shape.n_q * shape.head_dim, shape.n_kv * shape.head_dim
    b = 2
    wb = 0.5 + 1.0 / 32 if shape.mxfp4 else b
    per_layer_w = ((nq + 2 * nkv) * d + d * nq + 2 * F * d + d * F) * wb + 2 * d * b
    kv_read = 2 * shape.n_kv * (n_past + M) * shape.head_dim * b
    kv_write = 2 * M * nkv * b
    # the gate/up projection with the SwiGLU fused: both weight matrices, the normed input
    # (fp32, carried as its bf16 hi/lo pair) in, the SwiGLU output (likewise) out
    gate_up = 2 * F * d * wb + M * d * 4 + M * F * 4
    total = L * (per_layer_w + kv_read + kv_write) + V * d * b + V * 4 + d * b
    return {"step": total, "gate_up": gate_up, "weights": L * per_layer_w + V * d * b,
            "kv_read": L * kv_read}


def traffic_for_current_kernel():
    """HBM bytes per gate/up launch from the committed rocprofv3 counter runs, if they
    were taken on the current GEMM source (else null)."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        with open(GEMM_SRC, "rb") as f:
            h = hashlib.sha256(f.read()).hexdigest()[:16]
        if t.get("gemm_src_sha256_16") != h:
            return None
        return t.get("bytes_per_launch")
    except (OSError, ValueError):
        return None


def cpu_baseline(shape, seed: int, n_past: int, entry, n_layers: int) -> dict:
    """The oracle (fp64 C, OpenMP) on `n_layers` of the step's layers plus the LM head,
    scaled to the full step; input generation is not timed."""
    import numpy as np
    import oracle
    import synth
    sub = shape.with_layers(n_layers)
    w = oracle.Weights(sub, seed, cache_layers=True)
    for l in range(n_layers):
        w.layer(l)
    w.lm_head()
    w.final_norm()
    kv = oracle.KVState(sub, n_past + len(entry), seed=seed, n_synth=n_past)
    for l in range(n_layers):
        kv.layer(l)
    t0 = time.perf_counter()
    logits = oracle.forward(w, kv, n_past, entry)
    t_sample = time.perf_counter() - t0
    assert logits is not None and np.isfinite(logits).all()
    # split: LM head alone, to scale only the layers
    x_last = np.ones(shape.d_model)
    t1 = time.perf_counter()
    oracle.lib().orc_logits  # noqa: B018 (resolve before timing)
    import ctypes
    out = np.empty(shape.vocab)
    oracle.lib().orc_logits(ctypes.byref(oracle._cshape(sub)), oracle._p(x_last),
                            oracle._p(oracle._f32(w.final_norm())), oracle._p(oracle._f32(w.lm_head())),
                            None, oracle._p(out))
    t_lm = time.perf_counter() - t1
    t_layers = max(t_sample - t_lm, 1e-9)
    t_step = t_layers * shape.n_layers / n_layers + t_lm
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": len(entry) / t_step, "unit": "entry tok/s", "cores": cores, "kind": "oracle",
            "sample": f"{n_layers} of {shape.n_layers} layers + LM head of one step "
                      f"(timed {t_sample:.1f} s incl. LM head {t_lm:.2f} s), layers scaled x"
                      f"{shape.n_layers / n_layers:g}; est. step {t_step:.1f} s"}


def copy_calibration(mib: int) -> None:
    """Four launches of the library's copy kernel over `mib` MiB: each reads and writes
    exactly mib * 2^20 bytes, which calibrates FETCH_SIZE / WRITE_SIZE per byte."""
    import torch
    import paper_2606_29565_amd as spp
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(4):
        spp.copy_reference(dst, src, n)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_launch": n, "launches": 4}), flush=True)


def energy_reader():
    """A function returning the GPU's accumulated energy in J (amdsmi's energy counter of
    the device torch calls cuda:0), or None and the reason it is unavailable."""
    try:
        import amdsmi
        import torch
        amdsmi.amdsmi_init()
        handles = amdsmi.amdsmi_get_processor_handles()
        h = handles[0] if len(handles) == 1 else None
        if h is None:
            bus = getattr(torch.cuda.get_device_properties(0), "pci_bus_id", None)
            for c in handles:
                bdf = amdsmi.amdsmi_get_gpu_device_bdf(c)
                if bus is not None and int(bdf.split(":")[1], 16) == bus:
                    h = c
            if h is None:
                return None, f"{len(handles)} GPUs visible to amdsmi, none matched cuda:0"

        def read():
            e = amdsmi.amdsmi_get_energy_count(h)
            return e["energy_accumulator"] * e["counter_resolution"] * 1e-6

        read()
        return read, None
    except Exception as ex:  # reported, not fatal: the counter is a side measurement
        return None, f"{type(ex).__name__}: {ex}"


def energy_per_preposition(sess, entry, dist, stream, seconds: float = 3.0) -> dict:
    """Energy of back-to-back pre-positions for about `seconds`, against the idle draw
    over the same time (the counter's own clock), in J per pre-position."""
    import torch
    read, why = energy_reader()
    if read is None:
        return {"available": False, "reason": why}
    torch.cuda.synchronize()
    time.sleep(0.5)
    e0, t0 = read(), time.perf_counter()
    time.sleep(seconds)
    idle_w = (read() - e0) / (time.perf_counter() - t0)
    n = 0
    e0, t0 = read(), time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            sess.preposition(entry, dist, stream=stream)
        n += 20
        stream.synchronize()
    dt = time.perf_counter() - t0
    de = read() - e0
    return {"available": True, "prepositions": n, "seconds": dt, "busy_w": de / dt,
            "idle_w": idle_w, "j_per_preposition": de / n,
            "j_per_preposition_above_idle": (de - idle_w * dt) / n}


def idle_window(sess, entry, delta, dist, stream, n_past: int, cold_ms: float) -> dict:
    """The idle-window pass (spp_preposition_idle, one layer per chunk): its cost without
    a request against the plain pass, and what a request arriving mid-pass waits for:
    the time from setting the yield flag to the pass's return (device drained), and the
    cold request's latency measured from the flag."""
    import random
    import threading
    import paper_2606_29565_amd as spp
    flag = spp.YieldFlag()

    def wall(fn, k=5):
        ts = []
        for _ in range(k):
            sess.restore(n_past)
            stream.synchronize()
            t0 = time.perf_counter()
            fn()
            stream.synchronize()
            ts.append((time.perf_counter() - t0) * 1e3)
        return statistics.median(ts)

    plain_ms = wall(lambda: sess.preposition(entry, dist, stream=stream))
    idle_ms = wall(lambda: sess.preposition_idle(entry, dist, flag, 1, stream=stream))
    rng = random.Random(7)
    lat, req = [], []
    for _ in range(30):
        sess.restore(n_past)
        stream.synchronize()
        flag.clear()
        out = {}

        def run():
            out["r"] = sess.preposition_idle(entry, dist, flag, 1, stream=stream)
            out["t"] = time.perf_counter()

        th = threading.Thread(target=run)
        th.start()
        time.sleep(rng.uniform(0.0005, 0.8 * plain_ms * 1e-3))
        t_set = time.perf_counter()
        flag.set()
        th.join()
        if out["r"].status != spp.SPP_YIELDED:
            continue
        lat.append((out["t"] - t_set) * 1e3)
        sess.resume(entry + delta, dist, stream=stream)  # the request, on the cold path
        stream.synchronize()
        req.append((time.perf_counter() - t_set) * 1e3)
    lat.sort()
    req.sort()
    q = lambda v, f: v[min(len(v) - 1, int(len(v) * f))] if v else None  # noqa: E731
    return {"chunk_layers": 1, "plain_ms_wall": plain_ms, "idle_ms_wall": idle_ms,
            "yield_samples": len(lat), "yield_ms_p50": q(lat, 0.5), "yield_ms_max": q(lat, 1.0),
            "request_after_flag_ms_p50": q(req, 0.5), "request_after_flag_ms_max": q(req, 1.0),
            "cold_request_alone_ms": cold_ms}


def flush_mall(buf) -> None:
    """Write 512 MiB so that the distributions read next come from HBM, not the
    memory-side cache (256 MB on MI355X)."""
    import torch
    buf.fill_(1)
    torch.cuda.synchronize()


def gate_scans(vocab: int, fast_ids, tau: float, seed: int) -> dict:
    """The serve-time scan alone: one cached distribution (spp_gate) and 64 distributions
    with their own bitmaps (spp_gate_batch, 64 x vocab x 4 bytes), each warm (repeated)
    and MALL-cold (after a 512 MiB write).  Device time from events on the launch stream,
    end to end from the host clock.  The distributions belong to a 1-layer model with
    the same vocabulary (the scan reads only the distribution and the bitmap)."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    shape = synth.Shape("gatevocab", 1, 256, 4, 4, 64, 512, vocab, 1e4, "f32")
    w = synth.gpu_weights(shape, seed)
    model = spp.Model(1, 256, 4, 4, 64, 512, vocab, 1e4, False, w, max_tokens=16, max_sessions=64)
    stream = torch.cuda.current_stream()
    sessions, dists, readies, bms = [], [], [], []
    gen = torch.Generator(device="cuda").manual_seed(seed)
    bitmap = torch.from_numpy(synth.bitmap_from_ids(vocab, fast_ids)).cuda()
    for i in range(64):
        sess = spp.Session(model, 16)
        d = torch.empty(vocab, dtype=torch.float32, device="cuda")
        readies.append(sess.preposition([i + 1], d))
        sessions.append(sess)
        dists.append(d)
        bms.append(bitmap)
    torch.cuda.synchronize()
    for d in dists:  # realistic logits: N(0, 2), so the scan's branches behave as on a model
        d.normal_(0.0, 2.0, generator=gen)
    torch.cuda.synchronize()
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, cold, k=30):
        dev, wall = [], []
        for _ in range(k):
            if cold:
                flush_mall(flush)
            ev[0].record(stream)
            t0 = time.perf_counter()
            fn()
            t1 = time.perf_counter()
            ev[1].record(stream)
            ev[1].synchronize()
            dev.append(ev[0].elapsed_time(ev[1]) * 1e3)
            wall.append((t1 - t0) * 1e6)
        return statistics.median(dev), statistics.median(wall)

    one = lambda: spp.gate(readies[0], tau, bitmap, stream=stream)  # noqa: E731
    taus = [tau] * 64
    batch = lambda: spp.gate_batch(readies, taus, bms, stream=stream)  # noqa: E731
    one()
    batch()
    out = {}
    for name, fn, nbytes in (("single", one, vocab * 4), ("batch64", batch, 64 * vocab * 4)):
        for cold in (False, True):
            d_us, w_us = timed(fn, cold)
            out[f"{name}_{'cold' if cold else 'warm'}"] = {
                "device_us": round(d_us, 2), "e2e_us": round(w_us, 2),
                "gb_per_s_device": round(nbytes / (d_us * 1e-6) / 1e9, 1)}
    out["bytes_single"] = vocab * 4
    out["bytes_batch64"] = 64 * vocab * 4
    for sess in sessions:
        sess.close()
    del flush, model
    torch.cuda.empty_cache()
    return out


def cpu_baseline_one_core(shape, seed: int, n_past: int, entry, n_layers: int = 2) -> dict:
    """The same oracle on one thread (OpenMP limited to 1): `n_layers` layers scaled to the
    full depth, plus the LM head timed once."""
    import ctypes
    import numpy as np
    import oracle
    sub = shape.with_layers(n_layers)
    w = oracle.Weights(sub, seed, cache_layers=True)
    for l in range(n_layers):
        w.layer(l)
    w.lm_head()
    w.final_norm()
    kv = oracle.KVState(sub, n_past + len(entry), seed=seed, n_synth=n_past)
    for l in range(n_layers):
        kv.layer(l)
    gomp = ctypes.CDLL("libgomp.so.1")
    before = gomp.omp_get_max_threads()
    gomp.omp_set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.forward(w, kv, n_past, entry, logits=False)
        t = time.perf_counter() - t0
        out = np.empty(shape.vocab)
        x_last = np.ones(shape.d_model)
        t1 = time.perf_counter()
        oracle.lib().orc_logits(ctypes.byref(oracle._cshape(sub)), oracle._p(x_last),
                                oracle._p(oracle._f32(w.final_norm())),
                                oracle._p(oracle._f32(w.lm_head())), None, oracle._p(out))
        t_lm = time.perf_counter() - t1
    finally:
        gomp.omp_set_num_threads(before)
    assert np.isfinite(out).all()
    t_step = t * shape.n_layers / n_layers + t_lm
    return {"value": len(entry) / t_step, "unit": "entry tok/s", "cores": 1, "kind": "oracle",
            "sample": f"{n_layers} of {shape.n_layers} layers on one thread (timed {t:.1f} s), "
                      f"scaled x{shape.n_layers / n_layers:g}, plus the LM head ({t_lm:.2f} s); "
                      f"est. step {t_step:.0f} s"}


def copy_ceiling(mib: int = 1024) -> dict:
    """Achievable HBM bandwidth on this device: the library's plain copy kernel over
    `mib` MiB (read + write), median of 10."""
    import torch
    import paper_2606_29565_amd as spp
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ts = []
    for _ in range(11):
        ev[0].record(stream)
        spp.copy_reference(dst, src, n, stream=stream)
        ev[1].record(stream)
        ev[1].synchronize()
        ts.append(ev[0].elapsed_time(ev[1]))
    ms = statistics.median(ts[1:])
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_moved": 2 * n, "ms": ms, "gb_per_s": 2 * n / (ms * 1e-3) / 1e9}


def mxfp4_70b(steps: int, with_energy: bool = True) -> dict:
    """Secondary measurement: the pre-position of the 70B-shaped model with MXFP4
    projections (80 layers, d 8192, 64q/8kv x 128, SwiGLU 28672, vocab 128256, bf16
    LM head and cache), 8192 synthetic resident cells, a 24+8-token entry; device time
    of the pre-position (median over `steps`) and its per-kernel split."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    wl = synth.WORKLOADS["stream70b_mxfp4"]
    shape, seed, n_past, M = wl.shape, wl.seed, wl.n_past, wl.entry_len
    weights = synth.gpu_weights(shape, seed)
    model = spp.Model(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim,
                      shape.ffn, shape.vocab, shape.rope_base, True, weights, rms_eps=shape.eps,
                      max_tokens=M + 64, max_sessions=1, mxfp4=True)
    del weights  # the library keeps its own tiled copies
    cap = n_past + M + 64
    sess = spp.Session(model, cap)
    for l in range(shape.n_layers):
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(cap, l), shape, seed, 0, l, n_past)
    torch.cuda.synchronize()
    sess.restore(n_past)
    entry = synth.entry_tokens(wl, 0).tolist()
    dist = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(2):
        sess.preposition(entry, dist, stream=stream)
    ms = []
    for _ in range(steps):
        ev[0].record(stream)
        r = sess.preposition(entry, dist, stream=stream)
        ev[1].record(stream)
        ev[1].synchronize()
        if r.status != spp.SPP_OK:
            raise RuntimeError(f"pre-position status {r.status}")
        ms.append(ev[0].elapsed_time(ev[1]))
    pre_ms = statistics.median(ms)
    prof = model.profile_preposition(sess, entry, dist, stream=stream)
    ab = algorithmic_bytes(shape, M, n_past)
    gu_us, gu_n = prof["gemm_gate_up"]
    gu_avg = gu_us / max(gu_n, 1)
    sess.restore(n_past)
    energy = energy_per_preposition(sess, entry, dist, stream) if with_energy else None
    out = {"workload": "stream70b_mxfp4: 70B-shaped decoder, MXFP4 projections, n_s=8192, "
                       "entry 24+8=32 tokens",
           "preposition_ms_device": pre_ms, "entry_tok_s_device": M / (pre_ms * 1e-3),
           "step_algorithmic_gb": ab["step"] / 1e9,
           "step_hbm_frac": ab["step"] / (pre_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
           "gate_up_avg_launch_us": gu_avg,
           "gate_up_hbm_frac": ab["gate_up"] / (gu_avg * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "kernel_us_per_step": {k: round(v[0], 2) for k, v in prof.items()},
           "energy": energy}
    del sess, model
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no "
              "multi-GPU path; sessions would shard across GPUs with no exchange.", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.mxfp4_70b_only:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps({"mxfp4_70b": mxfp4_70b(args.steps, not args.no_energy)}), flush=True)
        return

    import numpy as np
    import torch
    import synth
    import paper_2606_29565_amd as spp

    wl = synth.WORKLOADS["stream8b"]
    shape, seed, n_past, M = wl.shape, wl.seed, wl.n_past, wl.entry_len
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    weights = synth.gpu_weights(shape, seed)
    model = spp.Model(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim,
                      shape.ffn, shape.vocab, shape.rope_base, True, weights, rms_eps=shape.eps,
                      max_tokens=M + 64, max_sessions=1)
    cap = n_past + M + 64  # room for a fall-through delta after the entry
    sess = spp.Session(model, cap)
    for l in range(shape.n_layers):
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(cap, l), shape, seed, 0, l, n_past)
    torch.cuda.synchronize()
    sess.restore(n_past)
    prefix = synth.cpu_tokens(24, seed, 1, shape.vocab).tolist()
    header = synth.cpu_tokens(8, seed, 2, shape.vocab).tolist()
    entry = prefix + header
    fast_ids = synth.fast_set(shape.vocab, wl.fast_set_size, seed)
    bitmap = torch.from_numpy(synth.bitmap_from_ids(shape.vocab, fast_ids)).to(dev)
    dist = torch.empty(shape.vocab, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    tau = 2.0

    def step():
        r = sess.preposition(entry, dist, stream=stream)
        if r.status != spp.SPP_OK:
            raise RuntimeError(f"pre-position status {r.status}")
        torch.cuda.current_stream().synchronize()  # the request arrives after the idle window
        outcome, tok, _ = spp.gate(r, tau, bitmap, stream=stream)
        sess.invalidate(spp.SPP_MUT_UPDATE)
        return outcome

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ms = []
    for _ in range(args.steps):
        ts = time.perf_counter()
        step()
        step_ms.append((time.perf_counter() - ts) * 1e3)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed / args.steps * 1e3
    step_ms.sort()
    pct = lambda f: step_ms[min(len(step_ms) - 1, int(len(step_ms) * f))]  # noqa: E731

    # device time of the pre-position alone (events on the same stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    pp_ms = []
    for _ in range(5):
        ev[0].record(stream)
        r = sess.preposition(entry, dist, stream=stream)
        ev[1].record(stream)
        ev[1].synchronize()
        pp_ms.append(ev[0].elapsed_time(ev[1]))
    pre_ms = statistics.median(pp_ms)

    # gate scan: end-to-end call latency on a decoded distribution (warm)
    torch.cuda.synchronize()
    gate_us = []
    for _ in range(200):
        g0 = time.perf_counter()
        spp.gate(r, tau, bitmap, stream=stream)
        gate_us.append((time.perf_counter() - g0) * 1e6)
    gate_us.sort()

    # critical-path latencies of one request, end to end on the host clock (median of 5):
    # cold (Eq. (lcold)): the whole realized input processed when the request arrives;
    # fall-through (Eq. (fallthrough)): entry pre-positioned, only the delta processed;
    # decode: one more token.  Each sample starts from n_past committed cells (restore).
    def request_ms(delta, pre_positioned):
        ts = []
        for _ in range(5):
            sess.restore(n_past)
            if pre_positioned:
                sess.preposition(entry, dist, stream=stream)
            stream.synchronize()
            t0 = time.perf_counter()
            sess.resume(delta if pre_positioned else entry + delta, dist, stream=stream)
            stream.synchronize()
            ts.append((time.perf_counter() - t0) * 1e3)
        return statistics.median(ts)

    delta8 = synth.cpu_tokens(8, seed, 6, shape.vocab).tolist()
    crit = {"cold_entry_plus_8_ms": request_ms(delta8, False),
            "fall_through_delta_8_ms": request_ms(delta8, True),
            "fall_through_delta_1_ms": request_ms(delta8[:1], True),
            "fast_path_gate_us_p50": None}
    dec = []
    for _ in range(5):
        sess.restore(n_past + 16)
        stream.synchronize()
        t0 = time.perf_counter()
        sess.resume(delta8[:1], dist, stream=stream)
        stream.synchronize()
        dec.append((time.perf_counter() - t0) * 1e3)
    crit["decode_step_ms"] = statistics.median(dec)

    # sliding-window shift (Sec. 3.6, the relocating mutation): the oldest 1024 of the 8192
    # committed cells dropped in every layer, the rest moved down with their keys turned
    shift_delta = 1024
    sh_ms = []
    for _ in range(3):
        sess.restore(n_past)
        ev[0].record(stream)
        sess.shift(shift_delta, stream=stream)
        ev[1].record(stream)
        ev[1].synchronize()
        sh_ms.append(ev[0].elapsed_time(ev[1]))
    sh_ms = statistics.median(sh_ms)
    # each moved cell's key and value read and written once, every layer and kv head
    sh_bytes = (shape.n_layers * shape.n_kv * (n_past - shift_delta) * shape.head_dim * 2 * 2 * 2)
    shift = {"cells": n_past, "delta": shift_delta, "ms_device": sh_ms,
             "algorithmic_gb": sh_bytes / 1e9, "gb_per_s": sh_bytes / (sh_ms * 1e-3) / 1e9}
    for l in range(shape.n_layers):  # the synthetic cells again, for what follows
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(cap, l), shape, seed, 0, l, n_past)
    torch.cuda.synchronize()
    sess.restore(n_past)

    # idle-window pass and its yield (Sec. 3.1), energy per pre-position (amdsmi)
    idle = idle_window(sess, entry, delta8, dist, stream, n_past, crit["cold_entry_plus_8_ms"])
    sess.restore(n_past)
    energy = None if args.no_energy else energy_per_preposition(sess, entry, dist, stream)
    sess.restore(n_past)

    # the serve-time scan alone (single and 64 distributions, warm and MALL-cold)
    scans = gate_scans(shape.vocab, fast_ids, tau, seed)
    ceiling = copy_ceiling()

    # per-kernel device time of one step (start and stop HIP events carried by each dispatch)
    prof = {}
    for _ in range(3):
        for k, (us, cnt) in model.profile_preposition(sess, entry, dist, stream=stream).items():
            a = prof.setdefault(k, [0.0, 0])
            a[0] += us
            a[1] += cnt
    gu_us, gu_n = prof["gemm_gate_up"]
    gu_avg_us = gu_us / max(gu_n, 1)
    ab = algorithmic_bytes(shape, M, n_past)
    achieved = ab["gate_up"] / (gu_avg_us * 1e-6) / 1e9
    traffic = traffic_for_current_kernel()

    out = {
        "metric": METRIC,
        "value": M * args.steps / elapsed,
        "unit": "entry tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "step_ms_p50_p90_p99": [pct(0.5), pct(0.9), pct(0.99)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random weights N(0,0.02), N(0,1) KV cells, uniform token ids)",
        "config": {"workload": "stream8b: 8B-shaped decoder (32 layers, d 4096, 32q/8kv x 128, "
                               "SwiGLU 14336, vocab 128256), persistent KV n_s=8192, entry 24+8=32 "
                               "tokens, gate tau=2 over a 64-token fast-answer set",
                   "n_past": n_past, "entry_len": M},
        "preposition_ms_device": pre_ms,
        "gate_us_e2e_p50": gate_us[len(gate_us) // 2],
        "critical_path": {**crit, "fast_path_gate_us_p50": gate_us[len(gate_us) // 2]},
        "gate_us_e2e_p99": gate_us[int(len(gate_us) * 0.99)],
        "shift": shift,
        "gate_scan": scans,
        "hbm_copy_ceiling": ceiling,
        "idle_window": idle,
        "energy": energy,
        "step_hbm_frac": ab["step"] / (pre_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "step_algorithmic_gb": ab["step"] / 1e9,
        "kernel_us_per_step": {k: round(v[0] / 3, 2) for k, v in prof.items()},
        "roofline": {"kernel": "gemm_gate_up", "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "avg_launch_us": gu_avg_us,
                     "algorithmic_bytes_per_launch": ab["gate_up"]},
    }
    if not args.no_mxfp4_70b:
        del sess, model, weights
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        out["mxfp4_70b"] = mxfp4_70b(5, not args.no_energy)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, seed, n_past, entry, args.cpu_layers)
        out["cpu_baseline_one_core"] = cpu_baseline_one_core(shape, seed, n_past, entry)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
