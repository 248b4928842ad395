"""Idle-window pre-position with a cooperative yield (Sec. 3.1: speculative work runs while
the session is idle and gives way to an arriving request; Alg. 1 otherwise unchanged).

Without a request the chunked pass must compute exactly what the plain pre-position
computes (same kernels, same order: bit-identical distributions), which the parity tests
already pin to the oracle; one case here is also checked against the oracle directly.
A yield must leave no trace: no ready record, n_s unchanged, and the next request's
result bit-identical to that of a session that never ran the yielded pass."""
import threading
import time

import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, fill_synthetic_kv, log, max_abs, oracle_logits, read_kv

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape("idle6", 6, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")
SEED = 31
TOL = 5e-2


def _dist(vocab):
    import torch
    return torch.empty(vocab, dtype=torch.float32, device="cuda")


@pytest.mark.parametrize("chunk", [1, 2, 4, 100])
def test_idle_pass_without_a_request_equals_the_plain_pass(chunk):
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    n_past, entry = 150, synth.cpu_tokens(20, SEED, 3, SHAPE.vocab).tolist()
    sess = spp.Session(b.model, n_past + 40)
    fill_synthetic_kv(b, sess, 0, n_past)
    sess.restore(n_past)
    d_plain, d_idle = _dist(SHAPE.vocab), _dist(SHAPE.vocab)
    r0 = sess.preposition(entry, d_plain)
    s0 = spp.ready_summary(r0)
    flag = spp.YieldFlag()
    r1 = sess.preposition_idle(entry, d_idle, flag, chunk_layers=chunk)
    assert r1.status == spp.SPP_OK
    torch.cuda.synchronize()
    assert torch.equal(d_plain, d_idle)
    s1 = spp.ready_summary(r1)
    assert (s1.argmax, s1.top1, s1.top2, s1.position) == (s0.argmax, s0.top1, s0.top2, s0.position)
    info = sess.info()
    assert info.valid == 1 and info.n_committed == n_past
    if chunk == 2:
        ref = oracle_logits(SHAPE, SEED, n_past, entry, kv_synth=True, last_only=True)
        err = max_abs(d_idle.cpu().numpy(), ref)
        log(f"idle pass, chunks of {chunk} layers: max|dlogit| vs oracle {err:.2e}")
        assert err <= TOL


def test_a_flag_already_set_yields_before_any_device_work():
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    n_past, entry = 100, synth.cpu_tokens(12, SEED, 4, SHAPE.vocab).tolist()
    sess = spp.Session(b.model, n_past + 40)
    fill_synthetic_kv(b, sess, 0, n_past)
    sess.restore(n_past)
    d = _dist(SHAPE.vocab)
    r_old = sess.preposition(entry, d)
    spp.ready_summary(r_old)
    torch.cuda.synchronize()
    kv_before = sess.kv.clone()
    flag = spp.YieldFlag()
    flag.set()
    e0 = sess.info().epoch
    r = sess.preposition_idle(entry, d, flag, chunk_layers=1)
    assert r.status == spp.SPP_YIELDED
    torch.cuda.synchronize()
    assert torch.equal(sess.kv, kv_before)  # nothing enqueued
    info = sess.info()
    assert info.valid == 0 and info.n_committed == n_past and info.epoch > e0
    assert spp.gate(r, 0.0, None)[0] == spp.SPP_FALL_INVALID
    assert spp.gate(r_old, 0.0, None)[0] == spp.SPP_FALL_INVALID  # replaced, not kept


def test_bad_idle_arguments_are_rejected():
    import paper_2606_29565_amd as spp
    b = build_model(SHAPE, SEED, max_tokens=32)
    sess = spp.Session(b.model, 64)
    d = _dist(SHAPE.vocab)
    flag = spp.YieldFlag()
    for chunk in (0, -3):
        with pytest.raises(spp.SppError):
            sess.preposition_idle([1, 2, 3], d, flag, chunk_layers=chunk)


@pytest.mark.timeout(300)
def test_a_request_arriving_mid_pass_makes_it_yield_without_a_trace():
    """The 8B shape (32 layers, 2048 resident cells): a thread sets the flag about 1 ms
    into the idle pass; the pass returns YIELDED within two layers' time, and the cold
    request that follows (entry + 8 tokens) gives the same distribution, bit for bit,
    as on a twin session that never ran the idle pass."""
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.M8B
    n_past, seed = 2048, 41
    b = build_model(shape, seed, max_tokens=64)
    entry = synth.cpu_tokens(32, seed, 1, shape.vocab).tolist()
    delta = synth.cpu_tokens(8, seed, 2, shape.vocab).tolist()
    sa, sb = spp.Session(b.model, n_past + 64), spp.Session(b.model, n_past + 64)
    for sess in (sa, sb):  # the same synthetic cells in both
        fill_synthetic_kv(b, sess, 0, n_past)
        sess.restore(n_past)
    torch.cuda.synchronize()
    d = _dist(shape.vocab)
    # warm: one full idle pass (also checks the no-request path at this shape)
    flag = spp.YieldFlag()
    assert sa.preposition_idle(entry, d, flag, chunk_layers=1).status == spp.SPP_OK
    sa.invalidate(spp.SPP_MUT_UPDATE)
    yielded = None
    for attempt in range(3):
        flag.clear()
        out = {}

        def idle():
            out["r"] = sa.preposition_idle(entry, d, flag, chunk_layers=1)
            out["t"] = time.perf_counter()

        th = threading.Thread(target=idle)
        th.start()
        time.sleep(0.001)
        t_set = time.perf_counter()
        flag.set()
        th.join()
        lat = (out["t"] - t_set) * 1e3
        log(f"attempt {attempt}: status {out['r'].status}, returned {lat:.3f} ms after the flag")
        if out["r"].status == spp.SPP_YIELDED:
            yielded = lat
            break
    assert yielded is not None, "the idle pass never saw the flag"
    assert yielded < 20.0
    info = sa.info()
    assert info.valid == 0 and info.n_committed == n_past
    assert spp.gate(out["r"], 0.0, None)[0] == spp.SPP_FALL_INVALID
    # the request: cold path over the entry and the delta, on both sessions
    da, db = _dist(shape.vocab), _dist(shape.vocab)
    sa.resume(entry + delta, da)
    sb.resume(entry + delta, db)
    torch.cuda.synchronize()
    assert torch.equal(da, db)
    K_a, V_a = read_kv(b, sa, 5, n_past + 40)
    K_b, V_b = read_kv(b, sb, 5, n_past + 40)
    np.testing.assert_array_equal(K_a, K_b)
    np.testing.assert_array_equal(V_a, V_b)
    log(f"yield after {yielded:.3f} ms; the cold request matches the twin session bit for bit")
