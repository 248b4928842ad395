"""The serve-time gate (Alg. 2, Eq. (gate)) on the GPU: the vocabulary scan against brute
force on planted distributions (spikes at the ends and at workgroup boundaries, exact
ties, NaN and infinities written into the cached distribution from the host), random
distributions over a tau sweep, and the batched scan over 64 distributions."""
import time

import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, log

pytestmark = pytest.mark.gpu

V8B = 128256


def _ready_session(vocab, seed=5, max_sessions=1):
    """A model whose ready records have `vocab` entries (tiny fp32 decoder)."""
    shape = synth.Shape("gatevocab", 1, 256, 4, 4, 64, 512, vocab, 1e4, "f32")
    b = build_model(shape, seed, max_tokens=16, max_sessions=max_sessions)
    return b, shape


def _decide(vals, tau, bitmap):
    s = oracle.summary(vals.astype(np.float64))
    return oracle.gate(True, True, s.nonfinite, s.gap, tau, oracle.in_bitmap(bitmap, s.argmax)), s


def _planted_cases(V, rng):
    cases = []
    base = rng.standard_normal(V).astype(np.float32)
    for i in (0, 1, V - 1, V - 2, 2047, 2048, 2049, 4095, 4096, V // 2):
        if i < V:
            v = base.copy()
            v[i] = 30.0
            cases.append((f"spike@{i}", v))
    v = base.copy(); v[[17, 9000 % V]] = 25.0; cases.append(("tie top1", v))
    v = base.copy(); v[5] = 25.0; v[[100 % V, 101 % V]] = 20.0; cases.append(("tie top2", v))
    v = base.copy(); v[7] = np.nan; cases.append(("nan", v))
    v = base.copy(); v[V - 1] = np.inf; cases.append(("+inf", v))
    v = base.copy(); v[3] = -np.inf; cases.append(("-inf", v))
    v = np.full(V, -1.5, np.float32); cases.append(("all equal", v))
    v = base.copy(); v[2048 % V] = 10.0; v[2049 % V] = 9.0; cases.append(("gap 1 at boundary", v))
    return cases


@pytest.mark.parametrize("V", [V8B, 4096, 1000, 97])
def test_gate_scan_planted_cases(V):
    import torch
    import paper_2606_29565_amd as spp
    b, shape = _ready_session(V)
    rng = np.random.default_rng(V)
    sess = spp.Session(b.model, 32)
    dist = torch.empty(V, dtype=torch.float32, device="cuda")
    r = sess.preposition([1, 2, 3], dist)
    torch.cuda.synchronize()
    for name, vals in _planted_cases(V, rng):
        ids = [int(np.nanargmax(np.where(np.isnan(vals), -np.inf, vals)))] if name != "all equal" else [0]
        for in_set in (True, False):
            bm = synth.bitmap_from_ids(V, ids if in_set else [])
            bm_dev = torch.from_numpy(bm).cuda()
            dist.copy_(torch.from_numpy(vals))
            torch.cuda.synchronize()
            for tau in (0.0, 0.5, 2.0, 4.9, 5.1):
                want, s = _decide(vals, tau, bm)
                out, tok, sc = spp.gate(r, tau, bm_dev)
                if not s.nonfinite:
                    assert sc.argmax == s.argmax, (name, sc.argmax, s.argmax)
                    assert sc.top1 == np.float32(s.top1) and sc.top2 == np.float32(s.top2)
                if abs(s.gap - tau) > 1e-4 or s.nonfinite:
                    assert out == want, (name, in_set, tau, out, want)
                if out == spp.SPP_SERVED:
                    assert tok == s.argmax
                else:
                    assert tok == -1
    sess.close()


def test_gate_random_distributions_tau_sweep():
    import torch
    import paper_2606_29565_amd as spp
    b, shape = _ready_session(V8B)
    sess = spp.Session(b.model, 32)
    dist = torch.empty(V8B, dtype=torch.float32, device="cuda")
    r = sess.preposition([4, 5], dist)
    rng = np.random.default_rng(0)
    fast = synth.fast_set(V8B, 64, 3)
    n = 0
    for trial in range(40):
        vals = (rng.standard_normal(V8B) * rng.uniform(0.3, 3)).astype(np.float32)
        if trial % 2:
            vals[fast[trial % 64]] = vals.max() + rng.uniform(0, 6)
        bm = synth.bitmap_from_ids(V8B, fast)
        dist.copy_(torch.from_numpy(vals))
        bm_dev = torch.from_numpy(bm).cuda()
        torch.cuda.synchronize()
        for tau in (0.5, 1.0, 2.0, 4.0):
            want, s = _decide(vals, tau, bm)
            out, tok, _ = spp.gate(r, tau, bm_dev)
            if abs(s.gap - tau) > 1e-4:
                assert out == want
                n += 1
    assert n >= 150
    sess.close()


def test_gate_batch_64_distributions_with_own_bitmaps():
    """Batched scan: 64 cached distributions, each with its own fast-answer bitmap."""
    import torch
    import paper_2606_29565_amd as spp
    b, shape = _ready_session(V8B, max_sessions=64)
    rng = np.random.default_rng(7)
    sessions, dists, readies, bms, vals_all = [], [], [], [], []
    for i in range(64):
        s = spp.Session(b.model, 16)
        d = torch.empty(V8B, dtype=torch.float32, device="cuda")
        readies.append(s.preposition([i + 1], d))
        sessions.append(s)
        dists.append(d)
    torch.cuda.synchronize()
    taus = []
    for i in range(64):
        vals = rng.standard_normal(V8B).astype(np.float32)
        top = int(rng.integers(0, V8B))
        vals[top] = vals.max() + float(rng.uniform(0, 5))
        if i % 7 == 0:
            vals[int(rng.integers(0, V8B))] = np.nan
        dists[i].copy_(torch.from_numpy(vals))
        ids = [top] if i % 3 else [int(rng.integers(0, V8B))]
        bm = synth.bitmap_from_ids(V8B, ids)
        bms.append(torch.from_numpy(bm).cuda())
        vals_all.append((vals, bm))
        taus.append(float(rng.choice([0.5, 1.0, 2.0, 4.0])))
    torch.cuda.synchronize()
    res = spp.gate_batch(readies, taus, bms)
    for i, (out, tok) in enumerate(res):
        want, s = _decide(vals_all[i][0], taus[i], vals_all[i][1])
        if abs(s.gap - taus[i]) > 1e-4 or s.nonfinite:
            assert out == want, (i, out, want)
        if out == spp.SPP_SERVED:
            assert tok == s.argmax
    for s in sessions:
        s.close()


def test_gate_latency_single_distribution():
    """End-to-end spp_gate latency on a decoded 128256-entry distribution (warm)."""
    import torch
    import paper_2606_29565_amd as spp
    b, shape = _ready_session(V8B)
    sess = spp.Session(b.model, 16)
    dist = torch.empty(V8B, dtype=torch.float32, device="cuda")
    r = sess.preposition([9], dist)
    bm = torch.from_numpy(synth.bitmap_from_ids(V8B, [1, 2, 3])).cuda()
    torch.cuda.synchronize()
    ts = []
    for _ in range(300):
        t0 = time.perf_counter()
        spp.gate(r, 2.0, bm)
        ts.append((time.perf_counter() - t0) * 1e6)
    ts.sort()
    log(f"gate e2e: p50 {ts[150]:.1f} us, p99 {ts[297]:.1f} us")
    assert ts[150] < 500.0
    sess.close()
