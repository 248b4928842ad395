"""spp_gate_batch_noalloc, the gate entry point that allocates nothing (its scan scratch is
a static device array of the library), against spp_gate_batch on the same handles: the
outcomes and tokens must be identical (integer decisions, bit-exact) and equal to Alg. 2
applied to the oracle's top-2 of each cached distribution, on two calls in a row -- 64
handles, then 5 -- and a call of more than 64 handles must be refused."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import log

pytestmark = pytest.mark.gpu

V = 128256


def _setup():
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.Shape("noalloc", 1, 256, 4, 4, 64, 512, V, 1e4, "f32")
    w = synth.gpu_weights(shape, 61)
    model = spp.Model(1, 256, 4, 4, 64, 512, V, 1e4, False, w, max_tokens=16, max_sessions=64)
    sessions, dists, readies = [], [], []
    for i in range(64):
        s = spp.Session(model, 16)
        d = torch.empty(V, dtype=torch.float32, device="cuda")
        readies.append(s.preposition([i + 1], d))
        sessions.append(s)
        dists.append(d)
    torch.cuda.synchronize()
    gen = torch.Generator(device="cuda").manual_seed(61)
    for i, d in enumerate(dists):
        d.normal_(0.0, 2.0, generator=gen)
        if i % 4 == 1:     # a clear winner at a block edge or the ends of the vocabulary
            d[[0, V - 1, 2048 * (i % 7), V // 2][i % 4]] = 30.0 + i
        elif i % 8 == 2:   # an exact tie for the top: gap 0, lowest index wins
            d[100 + i] = 25.0
            d[90000 + i] = 25.0
        elif i == 6:       # a NaN: never served
            d[777] = float("nan")
    torch.cuda.synchronize()
    return model, sessions, dists, readies


def _expected(dist, tau, bitmap):
    s = oracle.summary(dist.cpu().numpy().astype(np.float64))
    in_set = bitmap is not None and oracle.in_bitmap(bitmap, s.argmax) if not s.nonfinite else False
    out = oracle.gate(True, True, s.nonfinite, np.float32(s.top1) - np.float32(s.top2), tau, in_set)
    return out, (s.argmax if out == oracle.SERVED else -1)


def test_noalloc_gate_batch_matches_gate_batch_twice():
    import torch
    import paper_2606_29565_amd as spp
    model, sessions, dists, readies = _setup()
    rng = np.random.default_rng(61)
    bms_host, bms = [], []
    for i in range(64):
        if i % 5 == 4:
            bms_host.append(None)
            bms.append(None)
            continue
        top = int(torch.argmax(torch.nan_to_num(dists[i], nan=-1e30)))
        ids = rng.choice(V, 40, replace=False).tolist() + ([top] if i % 3 else [])
        bm = synth.bitmap_from_ids(V, ids)
        bms_host.append(bm)
        bms.append(torch.from_numpy(bm).cuda())
    sessions[9].invalidate(spp.SPP_MUT_UPDATE)   # a stale handle in the batch
    taus = [float(t) for t in rng.choice([0.0, 0.5, 2.0, 8.0, 40.0], 64)]
    a = spp.gate_batch(readies, taus, bms)
    b = spp.gate_batch(readies, taus, bms, noalloc=True)
    assert a == b
    for i in range(64):
        want = (spp.SPP_FALL_INVALID, -1) if i == 9 else _expected(dists[i], taus[i], bms_host[i])
        assert b[i] == want, (i, b[i], want)
    served = sum(o == spp.SPP_SERVED for o, _ in b)
    log(f"no-alloc gate, 64 handles: identical to spp_gate_batch, {served} served")
    assert 0 < served < 64
    # a second call right after, with a smaller input: 5 handles, other thresholds
    sub = [3, 17, 9, 40, 63]
    taus2 = [0.0, 1.0, 0.0, 3.0, 0.5]
    a2 = spp.gate_batch([readies[i] for i in sub], taus2, [bms[i] for i in sub])
    b2 = spp.gate_batch([readies[i] for i in sub], taus2, [bms[i] for i in sub], noalloc=True)
    assert a2 == b2
    for j, i in enumerate(sub):
        want = (spp.SPP_FALL_INVALID, -1) if i == 9 else _expected(dists[i], taus2[j], bms_host[i])
        assert b2[j] == want, (i, b2[j], want)
    # more handles than the static scratch covers: refused, nothing run
    with pytest.raises(spp.SppError) as ei:
        spp.gate_batch(readies + readies[:1], [0.0] * 65, bms + bms[:1], noalloc=True)
    assert ei.value.rc == spp.SPP_E_INVALID_ARG and "at most 64" in str(ei.value)
    for s in sessions:
        s.close()
    model.close()
