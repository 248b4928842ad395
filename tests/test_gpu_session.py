"""Session lifecycle on the GPU: Alg. 1's budget skip, the invalidation discipline of
Sec. 3.6 (stale handles after shift / rollback / update), Alg. 2's eligibility check, a
gate before the pre-position has finished, a random operation sequence with 1-in-8
mutations checked against the reference state machine and the oracle, and the batched
pre-position of several sessions of different lengths in one pass."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, fill_synthetic_kv, log, max_abs, oracle_logits, read_kv

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape("sess", 2, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")


def _mk(max_sessions=1, max_tokens=64):
    return build_model(SHAPE, 41, max_tokens=max_tokens, max_sessions=max_sessions)


def test_budget_skip_touches_nothing_and_invalidates():
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    sess = spp.Session(b.model, 64, budget=40)
    toks = synth.cpu_tokens(30, 41, 0, SHAPE.vocab).tolist()
    sess.append_delta(toks)
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    r_ok = sess.preposition([1, 2, 3], dist)
    assert r_ok.status == spp.SPP_OK
    torch.cuda.synchronize()
    before = sess.kv.clone()
    dist_before = dist.clone()
    r = sess.preposition(list(range(11)), dist)   # L = 11 > B = 40 - 30
    assert r.status == spp.SPP_SKIPPED_BUDGET
    torch.cuda.synchronize()
    assert torch.equal(sess.kv, before) and torch.equal(dist, dist_before)
    info = sess.info()
    assert info.valid == 0 and info.n_committed == 30 and info.used_cells == 30
    assert spp.gate(r_ok, 0.0, None)[0] == spp.SPP_FALL_INVALID
    r2 = sess.preposition(list(range(10)), dist)   # L = B is admitted
    assert r2.status == spp.SPP_OK and sess.info().position == 40


@pytest.mark.parametrize("kind,arg", [("shift", 0), ("rollback", 12), ("update", 0), ("append", 0),
                                      ("restore", 20), ("newpp", 0)])
def test_every_mutation_invalidates_the_handle(kind, arg):
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    sess = spp.Session(b.model, 64)
    sess.append_delta(synth.cpu_tokens(24, 41, 0, SHAPE.vocab).tolist())
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    r = sess.preposition([5, 6, 7], dist)
    summ = spp.ready_summary(r)
    bm = torch.from_numpy(synth.bitmap_from_ids(SHAPE.vocab, [summ.argmax])).cuda()
    assert spp.gate(r, 0.0, bm)[0] in (spp.SPP_SERVED, spp.SPP_FALL_GAP)
    e0 = sess.info().epoch
    if kind == "shift":
        sess.invalidate(spp.SPP_MUT_SHIFT)
    elif kind == "rollback":
        sess.invalidate(spp.SPP_MUT_ROLLBACK, arg)
        assert sess.info().n_committed == arg
    elif kind == "update":
        sess.invalidate(spp.SPP_MUT_UPDATE)
    elif kind == "append":
        sess.append_delta([9, 9])
        assert sess.info().n_committed == 26
    elif kind == "restore":
        sess.restore(arg)
    else:
        d2 = torch.empty_like(dist)
        sess.preposition([5, 6, 7], d2)
    info = sess.info()
    assert info.epoch > e0
    assert spp.gate(r, 0.0, bm)[0] == spp.SPP_FALL_INVALID
    with pytest.raises(spp.SppError):
        spp.ready_summary(r)


def test_eligibility_exact_match_and_relaxed_mode():
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    sess = spp.Session(b.model, 64)
    sess.append_delta(synth.cpu_tokens(16, 41, 0, SHAPE.vocab).tolist())
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    entry = [11, 12, 13, 14]
    r = sess.preposition(entry, dist)
    summ = spp.ready_summary(r)
    bm = torch.from_numpy(synth.bitmap_from_ids(SHAPE.vocab, [summ.argmax])).cuda()
    base = spp.gate(r, 0.0, bm)[0]
    assert spp.gate(r, 0.0, bm, realized=entry)[0] == base
    assert spp.gate(r, 0.0, bm, realized=[11, 12, 13, 15])[0] == spp.SPP_FALL_INELIGIBLE
    assert spp.gate(r, 0.0, bm, realized=entry + [1])[0] == spp.SPP_FALL_INELIGIBLE
    assert spp.gate(r, 0.0, bm, realized=entry[:3])[0] == spp.SPP_FALL_INELIGIBLE
    # the gate reads only: the record keeps serving
    assert spp.gate(r, 0.0, bm)[0] == base and sess.info().valid == 1
    with pytest.raises(spp.SppError):
        spp.gate(r, -1.0, bm)
    with pytest.raises(spp.SppError):
        spp.gate(r, float("nan"), bm)


def test_gate_before_the_preposition_finished_falls_through():
    """A request that arrives while the idle-window pass still runs is not served."""
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    sess = spp.Session(b.model, 64)
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        torch.cuda._sleep(200_000_000)   # a bounded spin ahead of the pre-position
        r = sess.preposition([1, 2, 3], dist, stream=side)
    assert sess.info().decoded == 0
    out, tok, _ = spp.gate(r, 0.0, None)
    assert out == spp.SPP_FALL_INVALID and tok == -1
    side.synchronize()
    assert sess.info().decoded == 1
    assert spp.gate(r, 0.0, None)[0] in (spp.SPP_FALL_NOT_IN_SET, spp.SPP_FALL_GAP)


def test_random_operations_with_one_in_eight_mutations():
    """Agentic schedule: after each pre-position a mutation arrives with probability 1/8
    before the request.  Flags and positions follow the reference state machine; a
    served token always equals the oracle's argmax of a fresh pass over the live
    sequence (the eligibility invariant of Sec. 3.6)."""
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    cap = 200
    sess = spp.Session(b.model, cap, budget=180)
    ref = oracle.SessionModel(180)
    rng = np.random.default_rng(8)
    ow = oracle.Weights(SHAPE, 41)
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    committed = []
    served = fell = mutated = 0
    bm_ids = set()
    for step in range(48):
        if len(committed) < 100 and rng.random() < 0.5:
            delta = synth.cpu_tokens(int(rng.integers(1, 12)), 41, 10 + step, SHAPE.vocab).tolist()
            sess.append_delta(delta)
            ref.update(delta)
            committed += delta
        entry = synth.cpu_tokens(int(rng.integers(1, 20)), 41, 100 + step, SHAPE.vocab).tolist()
        r = sess.preposition(entry, dist)
        st = ref.preposition(entry)
        assert (r.status == spp.SPP_SKIPPED_BUDGET) == (st == "SKIPPED")
        mutation = rng.random() < 1 / 8
        if mutation:
            mutated += 1
            kind = int(rng.integers(0, 3))
            if kind == 0:
                sess.invalidate(spp.SPP_MUT_SHIFT)
                ref.shift()
            elif kind == 1:
                n = int(rng.integers(0, len(committed) + 1))
                sess.invalidate(spp.SPP_MUT_ROLLBACK, n)
                ref.rollback(n)
                committed = committed[:n]
            else:
                delta = synth.cpu_tokens(3, 41, 500 + step, SHAPE.vocab).tolist()
                sess.append_delta(delta)
                ref.update(delta)
                committed += delta
        info = sess.info()
        assert (info.n_committed, info.used_cells, info.valid) == (ref.n_s, ref.used, int(ref.valid))
        if ref.valid:
            assert info.position == ref.position
        torch.cuda.synchronize()
        summ = spp.ready_summary(r) if ref.valid else None
        if summ is not None and step % 2 == 0:
            bm_ids.add(summ.argmax)
        bm = torch.from_numpy(synth.bitmap_from_ids(SHAPE.vocab, sorted(bm_ids))).cuda()
        out, tok, _ = spp.gate(r, 0.05, bm, realized=entry)
        if not ref.valid:
            assert out == spp.SPP_FALL_INVALID
            fell += 1
            continue
        if out == spp.SPP_SERVED:
            fresh = oracle.forward(ow, oracle.KVState(SHAPE, len(committed) + len(entry)), 0,
                                   committed + entry)
            s = oracle.summary(fresh)
            if s.gap > 0.1:
                assert tok == s.argmax
            served += 1
        else:
            fell += 1
    log(f"served {served}, fell through {fell}, mutated {mutated}")
    assert served > 0 and mutated > 0


def test_batched_preposition_matches_single_and_oracle():
    """Batched idle-window pre-positioning: sessions of different lengths (synthetic
    cells) and entries packed into one pass; one session over its budget is skipped."""
    import torch
    import paper_2606_29565_amd as spp
    b = _mk(max_sessions=8, max_tokens=160)
    rng = np.random.default_rng(5)
    specs = [(int(rng.integers(40, 600)), int(rng.integers(8, 40))) for _ in range(6)]
    specs.append((30, 50))   # over its budget of 60: skipped
    sessions, entries, dists = [], [], []
    for i, (n, L) in enumerate(specs):
        budget = 60 if i == 6 else 0
        s = spp.Session(b.model, n + L + 8, budget=budget)
        fill_synthetic_kv(b, s, i, n)
        s.restore(n)
        sessions.append(s)
        entries.append(synth.cpu_tokens(L, 41, 300 + i, SHAPE.vocab).tolist())
        dists.append(torch.zeros(SHAPE.vocab, dtype=torch.float32, device="cuda"))
    readies = spp.preposition_batch(sessions, entries, dists)
    torch.cuda.synchronize()
    assert [r.status for r in readies] == [spp.SPP_OK] * 6 + [spp.SPP_SKIPPED_BUDGET]
    assert float(dists[6].abs().max()) == 0.0
    for i in range(6):
        n, L = specs[i]
        got = dists[i].cpu().numpy()
        ref = oracle_logits(SHAPE, 41, n, entries[i], kv_synth=True, session=i)
        err = max_abs(got, ref)
        summ = spp.ready_summary(readies[i])
        s = oracle.summary(ref)
        log(f"batch session {i}: n={n} L={L} max|dlogit| {err:.2e}")
        assert err <= 5e-2
        if s.gap > 0.1:
            assert summ.argmax == s.argmax
        assert sessions[i].info().position == n + L
        # the same session pre-positioned alone gives the same distribution
        d1 = torch.empty_like(dists[i])
        sessions[i].preposition(entries[i], d1)
        torch.cuda.synchronize()
        assert max_abs(d1.cpu().numpy(), got) <= 2e-2


def test_capacity_beyond_the_limit_is_rejected():
    import torch
    import paper_2606_29565_amd as spp
    b = _mk()
    kv = torch.empty(64, dtype=torch.uint8, device="cuda")
    for cap in (0, spp.SPP_MAX_CAPACITY + 1):
        with pytest.raises(spp.SppError) as ei:
            spp.Session(b.model, cap, kv=kv)
        assert ei.value.rc == spp.SPP_E_INVALID_ARG and "capacity" in str(ei.value)
