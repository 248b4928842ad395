#!/usr/bin/env python3
"""Benchmark of the speculative pre-positioning hot path on one MI355X.

Headline workload (the larger-target configuration): a 32B-shaped decoder (64 layers,
d_model 5120, 64 query / 8 kv heads of dim 128, SwiGLU 27648, vocab 152064) in bf16
with seeded random weights, a persistent KV cache of n_s = 16384 synthetic cells, a
32-token entry, and an LM-head bias of 11 on one fast-answer token (decisive logits).

One step is the whole hot path: the pre-position (budget check, entry forward pass
over the resident cells with the in-place KV append, LM head with the fused
vocabulary reductions, ready record), the gate scan of the cached distribution
(tau = 2, a 64-token fast-answer set), and the invalidation of the record.
The cells are rewritten at the same positions each step (idempotent).

Legs reported beside it: the streaming 8B step (n_s = 8192, 24 + 8 entry tokens) with
its request latencies, idle-window yield, sliding-window shift and energy; the agentic
8B step (n_s = 32768, a 128-token envelope; attention against the matrix-core peak);
64 batched sessions of the 8B model (n_s ~ U[1024, 8192], entries ~ U[8, 64];
projections against the matrix-core peak); the gate scan alone; a 70B-shaped model
with MXFP4 projections.

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
MFMA_PEAK_TFS = 2500.0          # dense bf16 / fp16 matrix-core peak of the MI355X
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2606_29565_amd", "csrc")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=16,
                    help="decoder layers in the oracle's timed sample (scaled to the full step)")
    ap.add_argument("--no-mxfp4-70b", action="store_true",
                    help="skip the secondary measurement on the 70B-shaped MXFP4 model")
    ap.add_argument("--no-energy", action="store_true",
                    help="skip the energy measurements (seconds of back-to-back pre-positions)")
    ap.add_argument("--mxfp4-70b-only", action="store_true",
                    help="run only the 70B-shaped MXFP4 measurement and print its JSON")
    ap.add_argument("--legs", default="stream8b,agentic8b,batched8b,gate,mxfp4",
                    help="comma-separated legs to run beside the headline "
                         "(stream8b, agentic8b, batched8b, gate, mxfp4; empty for none)")
    ap.add_argument("--leg-only", default="",
                    help="run only this leg (headline, stream8b, agentic8b, batched8b, gate) and "
                         "print its JSON (for profiling one configuration)")
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
    act = lambda k, n: M * k * 4 + M * n * 4  # noqa: E731  (hi/lo in, fp32 or hi/lo out)
    per_kernel = {  # per step, the weight- and KV-streaming kernels
        "gemm_qkv": L * ((nq + 2 * nkv) * d * wb + act(d, nq + 2 * nkv)),
        "attention": L * (kv_read + M * nq * 2 + M * nq * 4),
        "gemm_o": L * (d * nq * wb + act(nq, d)),
        "gemm_gate_up": L * gate_up,
        "gemm_down": L * (d * F * wb + act(F, d)),
        "lm_head": V * d * b + V * 4,
    }
    return {"step": total, "gate_up": gate_up, "weights": L * per_layer_w + V * d * b,
            "kv_read": L * kv_read, "per_kernel": per_kernel}


def kernel_fractions(prof: dict, per_kernel: dict, passes: int) -> dict:
    """HBM fraction of 8 TB/s of every weight- and KV-streaming kernel class: its
    algorithmic bytes per step over its device time per step."""
    out = {}
    for k, nbytes in per_kernel.items():
        us = prof.get(k, (0.0, 0))[0] / passes
        if k == "attention":
            us += prof.get("attention_combine", (0.0, 0))[0] / passes
        if us > 0:
            out[k] = round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3)
    return out


def projection_flops(shape, rows: int, n_logit_rows: int) -> float:
    """Multiply-add flops (2 per product) of every projection of a pass over `rows` rows,
    plus the LM head over `n_logit_rows` decision points."""
    d, F, V, L = shape.d_model, shape.ffn, shape.vocab, shape.n_layers
    nq, nkv = shape.n_q * shape.head_dim, shape.n_kv * shape.head_dim
    per_row = L * ((nq + 2 * nkv) * d + d * nq + 2 * F * d + d * F)
    return 2.0 * rows * per_row + 2.0 * n_logit_rows * V * d


def attention_flops(shape, n_past: int, M: int) -> float:
    """Flops of the delta attention of a pass: every (query head, entry token j) against
    n_past + j + 1 keys, a QK dot product and a PV update of head_dim each."""
    keys = M * n_past + M * (M + 1) // 2
    return shape.n_layers * shape.n_q * keys * 4.0 * shape.head_dim


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the committed rocprofv3 counter
    runs (profiles/<kernel>_<workload>_traffic.json), if they were taken on the current
    source of that kernel (else null)."""
    try:
        with open(os.path.join(PROFILES, f"{kernel}_{workload}_traffic.json")) as f:
            t = json.load(f)
        with open(os.path.join(CSRC, t["source_file"]), "rb") as f:
            h = hashlib.sha256(f.read()).hexdigest()[:16]
        if t.get("source_sha256_16") != h:
            return None
        return t.get("bytes_per_launch")
    except (OSError, ValueError, KeyError):
        return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_gate_scan_ms(vocab: int) -> float:
    """The oracle's gate scan (its summary: a full sort for the top-2, log-sum-exp in
    double) over one distribution of `vocab` logits, median of 5."""
    import numpy as np
    import oracle
    v = np.random.default_rng(3).standard_normal(vocab) * 2.0
    ts = []
    for _ in range(5):
        t0 = time.perf_counter()
        oracle.summary(v)
        ts.append((time.perf_counter() - t0) * 1e3)
    return statistics.median(ts)


def cpu_baseline(shape, seed: int, n_past: int, entry, n_layers: int, bias=None) -> dict:
    """The oracle (fp64 C, OpenMP) on `n_layers` of the step's layers plus the LM head,
    scaled to the full step; input generation is not timed."""
    import numpy as np
    import oracle
    import synth
    sub = shape.with_layers(n_layers)
    w = oracle.Weights(sub, seed, lm_bias=bias, cache_layers=True)
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
    import ctypes as _ct
    cores = _ct.CDLL("libgomp.so.1").omp_get_max_threads()
    return {"value": len(entry) / t_step, "unit": "entry tok/s", "cores": cores, "kind": "oracle",
            "sample": f"{shape.name}: {n_layers} of {shape.n_layers} layers + LM head of one step "
                      f"(timed {t_sample:.1f} s incl. LM head {t_lm:.2f} s), layers scaled x"
                      f"{shape.n_layers / n_layers:g}; est. step {t_step:.1f} s",
            "cpu_model": cpu_model(), "ms_per_step_est": t_step * 1e3,
            "gate_scan_ms": oracle_gate_scan_ms(shape.vocab)}


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

    # the C calls with their arguments marshalled once (what a serving loop pays), and the
    # binding's per-call form (Python marshalling of 64 handles, taus and bitmaps included)
    taus = [tau] * 64
    one = spp.GateCall(readies[:1], [tau], [bitmap], stream=stream)
    batch = spp.GateCall(readies, taus, bms, stream=stream)
    one_py = lambda: spp.gate(readies[0], tau, bitmap, stream=stream)  # noqa: E731
    batch_py = lambda: spp.gate_batch(readies, taus, bms, stream=stream)  # noqa: E731
    one()
    batch()
    assert batch.outcomes() == batch_py() and one.outcomes()[0] == one_py()[:2]
    out = {}
    for name, fn, nbytes in (("single", one, vocab * 4), ("batch64", batch, 64 * vocab * 4)):
        for cold in (False, True):
            d_us, w_us = timed(fn, cold)
            out[f"{name}_{'cold' if cold else 'warm'}"] = {
                "device_us": round(d_us, 2), "e2e_us": round(w_us, 2),
                "gb_per_s_device": round(nbytes / (d_us * 1e-6) / 1e9, 1)}
    out["single_python_e2e_us"] = round(timed(one_py, False)[1], 2)
    out["batch64_python_e2e_us"] = round(timed(batch_py, False)[1], 2)
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
    # (at 32 rows the 4-bit gate/up runs unfused: its separate SwiGLU is counted in)
    sw_us = prof.get("swiglu", (0.0, 0))[0]
    gu_avg = (gu_us + sw_us) / max(gu_n, 1)
    sess.restore(n_past)
    energy = energy_per_preposition(sess, entry, dist, stream) if with_energy else None
    out = {"workload": "stream70b_mxfp4: 70B-shaped decoder, MXFP4 projections, n_s=8192, "
                       "entry 24+8=32 tokens",
           "preposition_ms_device": pre_ms, "entry_tok_s_device": M / (pre_ms * 1e-3),
           "step_algorithmic_gb": ab["step"] / 1e9,
           "step_hbm_frac": ab["step"] / (pre_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
           "gate_up_avg_launch_us": gu_avg,
           "gate_up_includes_swiglu_kernel": sw_us > 0,
           "gate_up_hbm_frac": ab["gate_up"] / (gu_avg * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "kernel_us_per_step": {k: round(v[0], 2) for k, v in prof.items()},
           "energy": energy}
    del sess, model
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def setup_session(shape, seed, n_past, M, bias=None, max_tokens=None, extra=64,
                  session_id=0):
    """A model of `shape` (seeded weights, optional LM-head bias) and one session with
    n_past synthetic resident cells, room for M + extra more."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    weights = synth.gpu_weights(shape, seed, bias)
    model = spp.Model(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim,
                      shape.ffn, shape.vocab, shape.rope_base, True, weights, rms_eps=shape.eps,
                      max_tokens=max_tokens or (M + 64), max_sessions=1)
    del weights  # the library keeps its own tiled copies of the projections
    cap = n_past + M + extra
    sess = spp.Session(model, cap)
    for l in range(shape.n_layers):
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(cap, l), shape, seed, session_id, l,
                          n_past)
    torch.cuda.synchronize()
    sess.restore(n_past)
    return model, sess, cap


def profile(model, sess, entry, dist, stream, passes=3):
    """Per-kernel device time summed over `passes` pre-positions (start and stop HIP events
    carried by each kernel's own dispatch, on the launch stream)."""
    prof = {}
    for _ in range(passes):
        for k, (us, cnt) in model.profile_preposition(sess, entry, dist, stream=stream).items():
            a = prof.setdefault(k, [0.0, 0])
            a[0] += us
            a[1] += cnt
    return prof


def device_ms(fn, stream, k=5):
    """Median device time of fn() on `stream` (events recorded around it)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ts = []
    for _ in range(k):
        ev[0].record(stream)
        fn()
        ev[1].record(stream)
        ev[1].synchronize()
        ts.append(ev[0].elapsed_time(ev[1]))
    return statistics.median(ts)


def roofline_of(prof, ab, passes, workload):
    """The dominant kernel's roofline entry (the fused gate/up + SwiGLU projection)."""
    gu_us, gu_n = prof["gemm_gate_up"]
    avg = gu_us / max(gu_n, 1)
    achieved = ab["gate_up"] / (avg * 1e-6) / 1e9
    return {"kernel": "gemm_gate_up", "bound": "hbm", "achieved": achieved,
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic_for("gemm_gate_up", workload), "avg_launch_us": avg,
            "algorithmic_bytes_per_launch": ab["gate_up"], "launches_timed": gu_n}


def leg_headline(steps, warmup) -> dict:
    """The 32B-shaped step: the timed loop of the headline value, its device time, the
    gate's latency, per-kernel times and fractions of the HBM roofline."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    wl = synth.WORKLOADS["target32b"]
    shape, seed, n_past, M = wl.shape, wl.seed, wl.n_past, wl.entry_len
    bias = synth.workload_bias(wl)
    model, sess, cap = setup_session(shape, seed, n_past, M, bias)
    entry = synth.entry_tokens(wl, 0).tolist()
    fast_ids = synth.fast_set(shape.vocab, wl.fast_set_size, seed)
    bitmap = torch.from_numpy(synth.bitmap_from_ids(shape.vocab, fast_ids)).cuda()
    dist = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    tau = 2.0
    outcomes = []

    def step():
        r = sess.preposition(entry, dist, stream=stream)
        if r.status != spp.SPP_OK:
            raise RuntimeError(f"pre-position status {r.status}")
        stream.synchronize()  # the request arrives after the idle window
        outcome, tok, _ = spp.gate(r, tau, bitmap, stream=stream)
        sess.invalidate(spp.SPP_MUT_UPDATE)
        return outcome

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    step_ms = []
    t0 = time.perf_counter()
    for _ in range(steps):
        ts = time.perf_counter()
        outcomes.append(step())
        step_ms.append((time.perf_counter() - ts) * 1e3)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms.sort()
    pct = lambda f: step_ms[min(len(step_ms) - 1, int(len(step_ms) * f))]  # noqa: E731
    pre_ms = device_ms(lambda: sess.preposition(entry, dist, stream=stream), stream)
    r = sess.preposition(entry, dist, stream=stream)
    torch.cuda.synchronize()
    gate_us = []
    for _ in range(200):
        g0 = time.perf_counter()
        spp.gate(r, tau, bitmap, stream=stream)
        gate_us.append((time.perf_counter() - g0) * 1e6)
    gate_us.sort()
    summ = spp.ready_summary(r)
    prof = profile(model, sess, entry, dist, stream)
    ab = algorithmic_bytes(shape, M, n_past)
    # the workload's decision points: entries 0..127 against the same resident cells, each
    # pre-positioned and gated at tau (outside the timed loop)
    gaps, served = [], 0
    for k in range(128):
        sess.invalidate(spp.SPP_MUT_UPDATE)
        rk = sess.preposition(synth.entry_tokens(wl, k).tolist(), dist, stream=stream)
        stream.synchronize()
        gaps.append(spp.ready_summary(rk).gap)
        served += spp.gate(rk, tau, bitmap, stream=stream)[0] == spp.SPP_SERVED
    sess.invalidate(spp.SPP_MUT_UPDATE)
    gs = sorted(gaps)
    decision_points = {"n": len(gaps), "gap_gt_tau_frac": sum(g > tau for g in gaps) / len(gaps),
                       "served_frac": served / len(gaps),
                       "gap_p10_p50_p90": [gs[len(gs) // 10], gs[len(gs) // 2], gs[len(gs) * 9 // 10]]}
    out = {
        "value": M * steps / elapsed, "ms_per_step": elapsed / steps * 1e3,
        "step_ms_p50_p90_p99": [pct(0.5), pct(0.9), pct(0.99)],
        "config": {"workload": "target32b: 32B-shaped decoder (64 layers, d 5120, 64q/8kv x 128, "
                               "SwiGLU 27648, vocab 152064), persistent KV n_s=16384, entry 32 "
                               "tokens, LM-head bias 10.1 on a fast-answer token, gate tau=2 over a "
                               "64-token fast-answer set",
                   "n_past": n_past, "entry_len": M},
        "preposition_ms_device": pre_ms,
        "gate_us_e2e_p50": gate_us[len(gate_us) // 2],
        "gate_us_e2e_p99": gate_us[int(len(gate_us) * 0.99)],
        "gate_outcomes": {spp.OUTCOME_NAMES[o]: outcomes.count(o) for o in set(outcomes)},
        "decision_gap": summ.gap,
        "decision_points": decision_points,
        "step_algorithmic_gb": ab["step"] / 1e9,
        "step_hbm_frac": ab["step"] / (pre_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "kernel_us_per_step": {k: round(v[0] / 3, 2) for k, v in prof.items()},
        "kernel_hbm_frac": kernel_fractions(prof, ab["per_kernel"], 3),
        "roofline": roofline_of(prof, ab, 3, "target32b"),
    }
    out["step_roofline"] = {"bound": "hbm", "achieved": ab["step"] / (pre_ms * 1e-3) / 1e9,
                            "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": out["step_hbm_frac"]}
    sess.close()
    model.close()
    del sess, model
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def leg_stream8b(steps, warmup, with_energy=True) -> dict:
    """The streaming 8B step with the request's critical path, the idle-window pass and its
    yield, the sliding-window shift and the energy per pre-position."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    wl = synth.WORKLOADS["stream8b"]
    shape, seed, n_past, M = wl.shape, wl.seed, wl.n_past, wl.entry_len
    model, sess, cap = setup_session(shape, seed, n_past, M)
    prefix = synth.cpu_tokens(24, seed, 1, shape.vocab).tolist()
    header = synth.cpu_tokens(8, seed, 2, shape.vocab).tolist()
    entry = prefix + header
    fast_ids = synth.fast_set(shape.vocab, wl.fast_set_size, seed)
    bitmap = torch.from_numpy(synth.bitmap_from_ids(shape.vocab, fast_ids)).cuda()
    dist = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    tau = 2.0

    def step():
        r = sess.preposition(entry, dist, stream=stream)
        stream.synchronize()
        spp.gate(r, tau, bitmap, stream=stream)
        sess.invalidate(spp.SPP_MUT_UPDATE)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / steps * 1e3
    pre_ms = device_ms(lambda: sess.preposition(entry, dist, stream=stream), stream)
    r = sess.preposition(entry, dist, stream=stream)
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
            "fast_path_gate_us_p50": gate_us[len(gate_us) // 2]}
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

    def shift_once():
        sess.restore(n_past)
        sess.shift(shift_delta, stream=stream)

    sh_ms = device_ms(shift_once, stream, k=3)
    # each moved cell's key and value read and written once, every layer and kv head
    sh_bytes = (shape.n_layers * shape.n_kv * (n_past - shift_delta) * shape.head_dim * 2 * 2 * 2)
    shift = {"cells": n_past, "delta": shift_delta, "ms_device": sh_ms,
             "algorithmic_gb": sh_bytes / 1e9, "gb_per_s": sh_bytes / (sh_ms * 1e-3) / 1e9}
    for l in range(shape.n_layers):  # the synthetic cells again, for what follows
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(cap, l), shape, seed, 0, l, n_past)
    torch.cuda.synchronize()
    sess.restore(n_past)
    idle = idle_window(sess, entry, delta8, dist, stream, n_past, crit["cold_entry_plus_8_ms"])
    sess.restore(n_past)
    energy = energy_per_preposition(sess, entry, dist, stream) if with_energy else None
    sess.restore(n_past)
    prof = profile(model, sess, entry, dist, stream)
    ab = algorithmic_bytes(shape, M, n_past)
    out = {"workload": "stream8b: 8B-shaped decoder (32 layers, d 4096, 32q/8kv x 128, SwiGLU "
                       "14336, vocab 128256), persistent KV n_s=8192, entry 24+8=32 tokens, gate "
                       "tau=2 over a 64-token fast-answer set",
           "entry_tok_s": M / (ms_per_step * 1e-3), "ms_per_step": ms_per_step,
           "preposition_ms_device": pre_ms,
           "gate_us_e2e_p50": gate_us[len(gate_us) // 2],
           "step_algorithmic_gb": ab["step"] / 1e9,
           "step_hbm_frac": ab["step"] / (pre_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
           "kernel_us_per_step": {k: round(v[0] / 3, 2) for k, v in prof.items()},
           "kernel_hbm_frac": kernel_fractions(prof, ab["per_kernel"], 3),
           "roofline": roofline_of(prof, ab, 3, "stream8b"),
           "critical_path": crit, "shift": shift, "idle_window": idle, "energy": energy}
    sess.close()
    model.close()
    del sess, model
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def leg_agentic8b() -> dict:
    """The agentic 8B step: a 128-token envelope against 32768 resident cells.  Its
    attention does 2.2 TFLOP per step, so it is reported against the matrix-core peak."""
    import torch
    import synth
    wl = synth.WORKLOADS["agentic8b"]
    shape, seed, n_past, M = wl.shape, wl.seed, wl.n_past, wl.entry_len
    model, sess, cap = setup_session(shape, seed, n_past, M)
    entry = synth.entry_tokens(wl, 0).tolist()
    dist = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(2):
        sess.preposition(entry, dist, stream=stream)
    pre_ms = device_ms(lambda: sess.preposition(entry, dist, stream=stream), stream)
    prof = profile(model, sess, entry, dist, stream)
    ab = algorithmic_bytes(shape, M, n_past)
    attn_us = prof["attention"][0] / 3
    comb_us = prof["attention_combine"][0] / 3
    fl = attention_flops(shape, n_past, M)
    proj_us = sum(prof[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")) / 3
    w_bytes = ab["weights"] - shape.vocab * shape.d_model * 2
    out = {"workload": "agentic8b: the 8B-shaped decoder, persistent KV n_s=32768, a 128-token "
                       "post-tool-call envelope appended delta-only",
           "preposition_ms_device": pre_ms, "entry_tok_s_device": M / (pre_ms * 1e-3),
           "step_algorithmic_gb": ab["step"] / 1e9,
           "attention_tflop": fl / 1e12,
           "attention_mfma_frac": fl / ((attn_us + comb_us) * 1e-6) / 1e12 / MFMA_PEAK_TFS,
           "attention_kv_hbm_frac": ab["kv_read"] / ((attn_us + comb_us) * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "projection_weights_hbm_frac": w_bytes / (proj_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "kernel_us_per_step": {k: round(v[0] / 3, 2) for k, v in prof.items()},
           "kernel_hbm_frac": kernel_fractions(prof, ab["per_kernel"], 3)}
    sess.close()
    model.close()
    del sess, model
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def leg_batched8b(steps: int = 5) -> dict:
    """64 sessions of the 8B model pre-positioned in one batched pass (n_s ~ U[1024, 8192],
    entries ~ U[8, 64]), then the 64 cached distributions gated in one batched scan.
    The projections carry ~2300 rows: reported against the matrix-core peak."""
    import torch
    import synth
    import paper_2606_29565_amd as spp
    wl = synth.WORKLOADS["batched8b"]
    shape, seed = wl.shape, wl.seed
    spec = synth.batched_spec(64, seed)
    total = sum(m for _, m in spec)
    weights = synth.gpu_weights(shape, seed)
    model = spp.Model(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim,
                      shape.ffn, shape.vocab, shape.rope_base, True, weights, rms_eps=shape.eps,
                      max_tokens=total, max_sessions=64)
    del weights
    sessions, entries, dists = [], [], []
    for i, (n, m) in enumerate(spec):
        s = spp.Session(model, n + m)
        for l in range(shape.n_layers):
            synth.gpu_fill_kv(s.kv.data_ptr(), model.kv_layout(n + m, l), shape, seed, i, l, n)
        s.restore(n)
        sessions.append(s)
        entries.append(synth.batched_entry(seed, i, m, shape.vocab).tolist())
        dists.append(torch.empty(shape.vocab, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    fast_ids = synth.fast_set(shape.vocab, wl.fast_set_size, seed)
    bitmap = torch.from_numpy(synth.bitmap_from_ids(shape.vocab, fast_ids)).cuda()
    spp.preposition_batch(sessions, entries, dists, stream=stream)
    pre_ms = device_ms(lambda: spp.preposition_batch(sessions, entries, dists, stream=stream),
                       stream, k=steps)
    readies = spp.preposition_batch(sessions, entries, dists, stream=stream)
    torch.cuda.synchronize()
    gate = spp.GateCall(readies, [2.0] * 64, [bitmap] * 64, stream=stream)
    g_us = []
    for _ in range(30):
        g0 = time.perf_counter()
        gate()
        g_us.append((time.perf_counter() - g0) * 1e6)
    prof = {}
    for k, (us, cnt) in spp.profile_preposition_batch(sessions, entries, dists, stream=stream).items():
        prof[k] = [us, cnt]
    proj_us = sum(prof[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down",
                                       "swiglu", "lm_head"))
    pf = projection_flops(shape, total, 64)
    kv_bytes = sum(shape.n_layers * 2 * shape.n_kv * (n + m) * shape.head_dim * 2 for n, m in spec)
    attn_us = prof["attention"][0] + prof["attention_combine"][0]
    w_bytes = algorithmic_bytes(shape, 1, 0)["weights"]
    out = {"workload": "batched8b: 64 sessions of the 8B-shaped decoder, n_s ~ U[1024, 8192], "
                       "entries ~ U[8, 64], one batched pre-position, one batched gate scan",
           "entry_rows": total, "preposition_ms_device": pre_ms,
           "entry_tok_s_device": total / (pre_ms * 1e-3),
           "projection_tflop": pf / 1e12,
           "projections_mfma_frac": pf / (proj_us * 1e-6) / 1e12 / MFMA_PEAK_TFS,
           "projections_mfma_frac_issued": 2 * pf / (proj_us * 1e-6) / 1e12 / MFMA_PEAK_TFS,
           "attention_kv_gb": kv_bytes / 1e9,
           "attention_hbm_frac": kv_bytes / (attn_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "weights_gb": w_bytes / 1e9,
           "gate_batch64_us_e2e_p50": statistics.median(g_us),
           "kernel_us_per_step": {k: round(v[0], 2) for k, v in prof.items()}}
    for s in sessions:
        s.close()
    model.close()
    del sessions, model
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
    import torch
    torch.cuda.set_device(0)
    if args.mxfp4_70b_only:
        print(json.dumps({"mxfp4_70b": mxfp4_70b(args.steps, not args.no_energy)}), flush=True)
        return
    if args.leg_only:
        import synth
        wl8 = synth.WORKLOADS["stream8b"]
        fn = {"headline": lambda: leg_headline(args.steps, args.warmup),
              "stream8b": lambda: leg_stream8b(args.steps, args.warmup, not args.no_energy),
              "agentic8b": leg_agentic8b, "batched8b": leg_batched8b,
              "gate": lambda: gate_scans(wl8.shape.vocab,
                                         synth.fast_set(wl8.shape.vocab, 64, wl8.seed), 2.0,
                                         wl8.seed)}[args.leg_only]
        print(json.dumps({args.leg_only: fn()}), flush=True)
        return
    legs = [x for x in args.legs.split(",") if x]

    head = leg_headline(args.steps, args.warmup)
    out = {
        "metric": METRIC,
        "value": head.pop("value"),
        "unit": "entry tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random weights N(0,0.02), N(0,1) KV cells, uniform token ids)",
    }
    out.update(head)
    print(json.dumps({"progress": "headline", "value": out["value"]}), file=sys.stderr, flush=True)
    if "stream8b" in legs:
        out["stream8b"] = leg_stream8b(args.steps, args.warmup, not args.no_energy)
        print('{"progress": "stream8b"}', file=sys.stderr, flush=True)
    if "agentic8b" in legs:
        out["agentic8b"] = leg_agentic8b()
        print('{"progress": "agentic8b"}', file=sys.stderr, flush=True)
    if "batched8b" in legs:
        out["batched8b"] = leg_batched8b()
        print('{"progress": "batched8b"}', file=sys.stderr, flush=True)
    if "gate" in legs:
        import synth
        wl = synth.WORKLOADS["stream8b"]
        out["gate_scan"] = gate_scans(wl.shape.vocab, synth.fast_set(wl.shape.vocab, 64, wl.seed),
                                      2.0, wl.seed)
        out["hbm_copy_ceiling"] = copy_ceiling()
        print('{"progress": "gate"}', file=sys.stderr, flush=True)
    if "mxfp4" in legs and not args.no_mxfp4_70b:
        out["mxfp4_70b"] = mxfp4_70b(5, not args.no_energy)
        print('{"progress": "mxfp4_70b"}', file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        import synth
        wl = synth.WORKLOADS["target32b"]
        entry = synth.entry_tokens(wl, 0)
        bias = synth.workload_bias(wl)
        out["cpu_baseline"] = cpu_baseline(wl.shape, wl.seed, wl.n_past, entry, args.cpu_layers,
                                           bias)
        out["cpu_baseline_one_core"] = cpu_baseline_one_core(wl.shape, wl.seed, wl.n_past, entry,
                                                             n_layers=1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
