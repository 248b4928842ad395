"""Gate calibration (Sec. 2.4) on decision points measured by the GPU gate scan.

The paper calibrates on (logit-gap, correctness) pairs of 128 decision points of its task
(Sec. 5), which need its data and trained model; seeded synthetic distributions stand in
for them here, with the paper's vocabulary-sized scan and a 31-token fast-answer set.
Each decision point has a ready distribution (noise plus an answer token raised by a
random margin) and a full-path distribution (the ready one moved by the realized
request).  The GPU scan gives each point's argmax, gap and set bit, and the argmax of its
full-path distribution; the oracle computes the same from the same values.  The
calibration curves and the selected threshold must be identical."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, log

pytestmark = pytest.mark.gpu

V = 128256
N_POINTS = 128
TAUS = np.arange(0.0, 6.0001, 0.25)


def _points(rng, fast):
    """Seeded synthetic (ready, full) logit pairs whose oracle gaps keep clear of every
    threshold of the sweep, so fp32 and fp64 gaps fall on the same side of each."""
    pts = []
    while len(pts) < N_POINTS:
        noise = rng.standard_normal(V).astype(np.float32)
        ans = int(fast[rng.integers(len(fast))]) if rng.uniform() < 0.85 else int(rng.integers(V))
        ready = noise.copy()
        ready[ans] = np.float32(noise.max() + rng.uniform(-0.5, 6.5))
        full = (ready + rng.normal(0.0, 0.8, V)).astype(np.float32)
        g = oracle.summary(ready.astype(np.float64)).gap
        if np.min(np.abs(g - TAUS)) > 1e-3:
            pts.append((ready, full))
    return pts


def test_calibration_from_gpu_scans_matches_the_oracle():
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.Shape("calib", 1, 256, 4, 4, 64, 512, V, 1e4, "f32")
    b = build_model(shape, 3, max_tokens=16)
    sess = spp.Session(b.model, 32)
    dist = torch.empty(V, dtype=torch.float32, device="cuda")
    r = sess.preposition([1, 2, 3], dist)
    torch.cuda.synchronize()
    fast = synth.fast_set(V, 31, 9)
    bitmap_np = synth.bitmap_from_ids(V, fast.tolist())
    bitmap = torch.from_numpy(bitmap_np).cuda()
    rng = np.random.default_rng(2026)
    pts = _points(rng, fast)
    g_gpu, a_gpu, c_gpu = [], [], []
    g_orc, a_orc, c_orc = [], [], []
    for ready, full in pts:
        dist.copy_(torch.from_numpy(ready))
        _, _, s = spp.gate(r, 0.0, bitmap)
        dist.copy_(torch.from_numpy(full))
        _, _, sf = spp.gate(r, 0.0, bitmap)
        g_gpu.append(s.gap)
        a_gpu.append(1 if (s.flags >> 1) & 1 else 0)
        c_gpu.append(1 if sf.argmax == s.argmax else 0)
        so = oracle.summary(ready.astype(np.float64))
        sfo = oracle.summary(full.astype(np.float64))
        assert so.argmax == s.argmax and sfo.argmax == sf.argmax
        g_orc.append(so.gap)
        a_orc.append(1 if oracle.in_bitmap(bitmap_np, so.argmax) else 0)
        c_orc.append(1 if sfo.argmax == so.argmax else 0)
    assert a_gpu == a_orc and c_gpu == c_orc
    for r_max in (0.05, 0.1, 0.15, 0.25):
        star, curve = spp.gate_calibrate(g_gpu, a_gpu, c_gpu, r_max, taus=TAUS)
        ostar, ocurve = oracle.calibrate(g_orc, a_orc, c_orc, r_max, taus=TAUS)
        assert star == ostar
        assert [(p.served, p.wrong) for p in curve] == [(c[1], c[2]) for c in ocurve]
    star, curve = spp.gate_calibrate(g_gpu, a_gpu, c_gpu, 0.15, taus=TAUS)
    at2 = curve[list(TAUS).index(2.0)]
    log(f"synthetic calibration, {N_POINTS} points: tau* = {star} for r_max 0.15; at tau 2: "
        f"coverage {at2.coverage:.3f} [{at2.coverage_lo:.3f}, {at2.coverage_hi:.3f}], "
        f"false-accept {at2.risk:.3f} [{at2.risk_lo:.3f}, {at2.risk_hi:.3f}]")
