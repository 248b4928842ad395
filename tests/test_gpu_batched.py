"""Batched idle-window pre-positioning at its real configuration: 64 sessions of the
8B shape (d 4096, 32/8 heads of 128, SwiGLU 14336, vocab 128256; two layers), each with
U[1024, 8192] synthetic resident cells and an entry of U[8, 64] tokens, packed into one
pass through spp_preposition_batch (Alg. 1 per session).  Every logit of every session
is compared with the oracle's pass over that session alone.  Also: a model whose
max_sessions is smaller than the batch splits it into passes of at most max_sessions
decision points, each distribution equal to the session's own pre-position."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, fill_synthetic_kv, log, max_abs

pytestmark = pytest.mark.gpu

LOGIT_TOL = 5e-2


@pytest.mark.timeout(900)
def test_batched64_real_configuration_every_logit():
    import torch
    import paper_2606_29565_amd as spp
    wl = synth.WORKLOADS["batched8b"]
    shape = wl.shape.with_layers(2)
    seed = wl.seed
    spec = synth.batched_spec(64, seed)
    total = sum(m for _, m in spec)
    log(f"batched8b: 64 sessions, {total} entry rows, n_s in [{min(n for n, _ in spec)}, "
        f"{max(n for n, _ in spec)}]")
    b = build_model(shape, seed, max_tokens=total, max_sessions=64)
    sessions, entries, dists = [], [], []
    for i, (n, m) in enumerate(spec):
        s = spp.Session(b.model, n + m)
        fill_synthetic_kv(b, s, i, n)
        s.restore(n)
        sessions.append(s)
        entries.append(synth.batched_entry(seed, i, m, shape.vocab).tolist())
        dists.append(torch.empty(shape.vocab, dtype=torch.float32, device="cuda"))
    readies = spp.preposition_batch(sessions, entries, dists)
    torch.cuda.synchronize()
    assert all(r.status == spp.SPP_OK for r in readies)
    got = [d.cpu().numpy().astype(np.float64) for d in dists]
    summs = [spp.ready_summary(r) for r in readies]
    for s in sessions:
        s.close()
    b.model.close()
    del b, dists
    torch.cuda.empty_cache()
    w = oracle.Weights(shape, seed, cache_layers=True)
    worst = 0.0
    for i, (n, m) in enumerate(spec):
        kv = oracle.KVState(shape, n + m, seed=seed, session=i, n_synth=n)
        ref = oracle.forward(w, kv, n, entries[i], last_only=True)
        err = max_abs(got[i], ref)
        worst = max(worst, err)
        s = oracle.summary(ref)
        if i % 8 == 0 or err > LOGIT_TOL:
            log(f"session {i}: n_s={n} M={m} max|dlogit| {err:.2e}")
        assert err <= LOGIT_TOL, (i, err)
        if s.gap > 0.1:
            assert summs[i].argmax == s.argmax, (i, summs[i].argmax, s.argmax)
        assert summs[i].position == n + m
    log(f"batched8b: worst max|dlogit| over 64 sessions {worst:.2e}")


def test_batch_larger_than_max_sessions_takes_several_passes():
    """max_sessions = 2 and 5 sessions: passes of at most 2 decision points, each
    distribution equal to that session's own pre-position and within the bar of the
    oracle."""
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.Shape("sess", 2, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")
    b = build_model(shape, 43, max_tokens=64, max_sessions=2)
    sessions, entries, dists = [], [], []
    for i in range(5):
        n = 20 + 7 * i
        s = spp.Session(b.model, n + 16)
        fill_synthetic_kv(b, s, i, n)
        s.restore(n)
        sessions.append(s)
        entries.append(synth.cpu_tokens(3 + i, 43, 50 + i, shape.vocab).tolist())
        dists.append(torch.empty(shape.vocab, dtype=torch.float32, device="cuda"))
    readies = spp.preposition_batch(sessions, entries, dists)
    torch.cuda.synchronize()
    assert [r.status for r in readies] == [spp.SPP_OK] * 5
    w = oracle.Weights(shape, 43)
    for i in range(5):
        got = dists[i].cpu().numpy()
        n = 20 + 7 * i
        kv = oracle.KVState(shape, n + len(entries[i]), seed=43, session=i, n_synth=n)
        ref = oracle.forward(w, kv, n, entries[i])
        assert max_abs(got, ref) <= LOGIT_TOL, (i, max_abs(got, ref))
        d1 = torch.empty_like(dists[i])
        sessions[i].preposition(entries[i], d1)
        torch.cuda.synchronize()
        assert max_abs(d1.cpu().numpy(), got) <= 2e-2
    for s in sessions:
        s.close()
    b.model.close()
