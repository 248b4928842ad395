"""Fall-through resume on the GPU (Eq. (fallthrough), Sec. 3.5): after a pre-position the
request extends the entry by a delta; the entry cells stay in place (constant-time
restore) and only the delta is processed.  Each ready distribution must equal the
oracle's fresh forward pass over the whole live sequence (the eligibility invariant of
Sec. 3.6 applied to the resumed state), the cells written by the pre-position and by the
resume must equal the oracle's, and the session must follow the reference state model."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, log, max_abs, read_kv

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape("resume", 2, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")
SEED = 43
TOL = 5e-2  # max |dlogit| bar of the pre-position path


def _fresh(tokens, kv_out=None):
    """The oracle's logits at the last of `tokens`, forward pass from position 0."""
    w = oracle.Weights(SHAPE, SEED, cache_layers=True)
    kv = oracle.KVState(SHAPE, len(tokens))
    out = oracle.forward(w, kv, 0, list(tokens))
    if kv_out is not None:
        kv_out.append(kv)
    return out


def _toks(n, stream):
    return synth.cpu_tokens(n, SEED, stream, SHAPE.vocab).tolist()


def _dist():
    import torch
    return torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")


def test_resume_keeps_entry_cells_and_matches_fresh_pass():
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    sess = spp.Session(b.model, 96)
    committed, entry, delta = _toks(20, 1), _toks(8, 2), _toks(5, 3)
    sess.append_delta(committed)
    d0, d1 = _dist(), _dist()
    r0 = sess.preposition(entry, d0)
    r1 = sess.resume(delta, d1)
    assert r1.status == spp.SPP_OK
    torch.cuda.synchronize()
    info = sess.info()
    assert (info.n_committed, info.used_cells, info.valid, info.position, info.entry_len) == \
        (33, 33, 1, 33, 0)
    # the entry's ready record is consumed: its handle is stale
    assert spp.gate(r0, 0.0, None)[0] == spp.SPP_FALL_INVALID
    with pytest.raises(spp.SppError):
        spp.ready_summary(r0)
    kvs = []
    ref = _fresh(committed + entry + delta, kvs)
    got = d1.cpu().numpy()
    err = max_abs(got, ref)
    s_ref = oracle.summary(ref)
    summ = spp.ready_summary(r1)
    log(f"resume: max|dlogit| {err:.2e}, oracle gap {s_ref.gap:.3f}")
    assert err <= TOL
    assert summ.position == 33
    if s_ref.gap > 0.1:
        assert summ.argmax == s_ref.argmax
    # every cell: the committed ones, the entry's (written by the pre-position) and the
    # delta's (written by the resume)
    for layer in range(SHAPE.n_layers):
        K, V = read_kv(b, sess, layer, 33)
        Kr, Vr = kvs[0].layer(layer)
        Kr, Vr = np.asarray(Kr)[:, :33], np.asarray(Vr)[:, :33]
        assert np.allclose(K, Kr, atol=4e-2, rtol=2.0 ** -7)
        assert np.allclose(V, Vr, atol=4e-2, rtol=2.0 ** -7)
    # the relaxed gate may serve from the resumed record
    bm = torch.from_numpy(synth.bitmap_from_ids(SHAPE.vocab, [summ.argmax])).cuda()
    out, tok, _ = spp.gate(r1, 0.0, bm)
    assert out in (spp.SPP_SERVED, spp.SPP_FALL_GAP)
    assert spp.gate(r1, 0.0, bm, realized=entry)[0] == spp.SPP_FALL_INELIGIBLE


def test_greedy_decode_steps_follow_the_oracle():
    """A one-token resume is a decode step: four greedy steps after a fall-through."""
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    sess = spp.Session(b.model, 96)
    seq = _toks(30, 4)
    sess.append_delta(seq)
    entry = _toks(6, 5)
    d = _dist()
    sess.preposition(entry, d)
    seq = seq + entry
    r = sess.resume(_toks(2, 6), d)
    seq = seq + _toks(2, 6)
    for step in range(4):
        torch.cuda.synchronize()
        ref = _fresh(seq)
        err = max_abs(d.cpu().numpy(), ref)
        summ = spp.ready_summary(r)
        s_ref = oracle.summary(ref)
        log(f"decode step {step}: max|dlogit| {err:.2e}, oracle gap {s_ref.gap:.3f}")
        assert err <= TOL and summ.position == len(seq)
        if s_ref.gap > 0.1:
            assert summ.argmax == s_ref.argmax
        tok = s_ref.argmax  # follow the oracle's token so both sides stay on one sequence
        r = sess.resume([tok], d)
        seq = seq + [tok]
    assert sess.info().n_committed == len(seq)


def test_resume_without_entry_is_the_cold_path():
    """A mutation drops the entry cells; the resume then appends the delta after the
    committed cells (the request re-supplies the entry itself)."""
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    sess = spp.Session(b.model, 96)
    committed, entry = _toks(17, 7), _toks(9, 8)
    sess.append_delta(committed)
    d = _dist()
    sess.preposition(entry, d)
    sess.invalidate(spp.SPP_MUT_SHIFT)
    assert sess.info().used_cells == 17
    r = sess.resume(entry + [3, 4], d)
    torch.cuda.synchronize()
    ref = _fresh(committed + entry + [3, 4])
    assert max_abs(d.cpu().numpy(), ref) <= TOL
    assert spp.ready_summary(r).position == 28 and sess.info().n_committed == 28


def test_long_delta_is_processed_in_chunks():
    """A delta longer than max_tokens runs as several passes; only the last one writes
    the distribution."""
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=16)
    sess = spp.Session(b.model, 128)
    committed, entry, delta = _toks(10, 9), _toks(12, 10), _toks(40, 11)
    sess.append_delta(committed)
    d = _dist()
    sess.preposition(entry, d)
    r = sess.resume(delta, d)
    torch.cuda.synchronize()
    ref = _fresh(committed + entry + delta)
    err = max_abs(d.cpu().numpy(), ref)
    log(f"chunked resume (40 tokens, max_tokens 16): max|dlogit| {err:.2e}")
    assert err <= TOL and spp.ready_summary(r).position == 62


def test_resume_beyond_capacity_changes_nothing():
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    sess = spp.Session(b.model, 40, budget=30)
    sess.append_delta(_toks(10, 12))
    d = _dist()
    r = sess.preposition(_toks(20, 13), d)
    ref = oracle.SessionModel(30, cells=40)
    ref.update(_toks(10, 12))
    ref.preposition(_toks(20, 13))
    before = sess.info()
    with pytest.raises(spp.SppError):
        sess.resume(_toks(11, 14), d)
    assert ref.resume(_toks(11, 14)) == "CAPACITY"
    after = sess.info()
    assert (after.n_committed, after.used_cells, after.valid, after.epoch) == \
        (before.n_committed, before.used_cells, before.valid, before.epoch)
    torch.cuda.synchronize()
    assert spp.gate(r, 0.0, None)[0] != spp.SPP_FALL_INVALID  # the entry record is intact
    # the budget bounds pre-positions only: a resume may use the cells beyond it
    r2 = sess.resume(_toks(10, 15), d)
    assert ref.resume(_toks(10, 15)) == "OK"
    info = sess.info()
    assert (info.n_committed, info.used_cells, info.valid, info.position) == \
        (ref.n_s, ref.used, int(ref.valid), ref.position) == (40, 40, 1, 40)
    assert r2.status == spp.SPP_OK
