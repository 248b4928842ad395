"""Sliding-window shift (Sec. 3.6, the mutation that relocates positions) on the GPU,
checked against the oracle: the oldest cells are dropped, the others move down with their
keys turned back by the shift (rotate-half RoPE) and their values unchanged, and the
ready distribution is invalidated in the same call.

Kernel parity uses the seeded synthetic cells, which both sides generate independently,
so the inputs are identical: values must move bit for bit and keys may differ by one
bf16 rounding (the GPU turns them in fp32, the oracle in fp64).  End-to-end parity runs a
real prefill on both sides, shifts, pre-positions an entry and compares the logits."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_model, fill_synthetic_kv, log, max_abs, read_kv

pytestmark = pytest.mark.gpu

BF16 = synth.Shape("shiftb", 2, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")
SEED = 23
TOL = 5e-2


def _oracle_kv_after_shift(shape, seed, n, delta, cap):
    kv = oracle.KVState(shape, cap, seed=seed, session=0, n_synth=n)
    oracle.shift_cells(shape, kv, n, delta)
    return kv


def _key_close(got, want, bf16):
    # one rounding of the cache format apart (the GPU turns keys in fp32, the oracle in fp64)
    rtol = 2.0 ** -7 if bf16 else 2.0 ** -22
    return np.allclose(got, want, rtol=rtol, atol=1e-5)


@pytest.mark.parametrize("shape_name,n,delta", [
    ("bf16", 300, 1), ("bf16", 300, 63), ("bf16", 300, 64), ("bf16", 300, 65),
    ("bf16", 300, 257), ("bf16", 300, 299), ("f32", 200, 37), ("f32", 129, 128)])
def test_shift_moves_and_turns_the_cells_like_the_oracle(shape_name, n, delta):
    import torch
    import paper_2606_29565_amd as spp
    shape = BF16 if shape_name == "bf16" else synth.TINY
    b = build_model(shape, SEED, max_tokens=32)
    cap = n + 40
    sess = spp.Session(b.model, cap)
    fill_synthetic_kv(b, sess, 0, n)
    sess.restore(n)
    e0 = sess.info().epoch
    sess.shift(delta)
    torch.cuda.synchronize()
    info = sess.info()
    assert info.n_committed == n - delta and info.valid == 0 and info.epoch == e0 + 1
    okv = _oracle_kv_after_shift(shape, SEED, n, delta, cap)
    n_new = n - delta
    for l in range(shape.n_layers):
        K, V = read_kv(b, sess, l, n_new)
        Ko, Vo = okv.layer(l)
        np.testing.assert_array_equal(V, Vo[:, :n_new])
        assert _key_close(K, Ko[:, :n_new], shape.bf16), \
            f"layer {l}: keys differ by {max_abs(K, Ko[:, :n_new]):.3e}"
    log(f"shift {shape_name} n={n} delta={delta}: cells match the oracle")


def test_shift_then_preposition_matches_the_oracle():
    import torch
    import paper_2606_29565_amd as spp
    seed, n, delta, L = 67, 180, 70, 12
    b = build_model(BF16, seed, max_tokens=64)
    toks = synth.cpu_tokens(n + L, seed, 0, BF16.vocab).tolist()
    sess = spp.Session(b.model, n + L + 8)
    sess.append_delta(toks[:n])
    sess.shift(delta)
    dist = torch.empty(BF16.vocab, dtype=torch.float32, device="cuda")
    r = sess.preposition(toks[n:], dist)
    torch.cuda.synchronize()
    assert sess.info().position == n - delta + L
    w = oracle.Weights(BF16, seed, cache_layers=True)
    kv = oracle.KVState(BF16, n + L + 8)
    oracle.forward(w, kv, 0, toks[:n], logits=False)
    oracle.shift_cells(BF16, kv, n, delta)
    ref = oracle.forward(w, kv, n - delta, toks[n:])
    got = dist.cpu().numpy()
    err = max_abs(got, ref)
    s_ref = oracle.summary(ref)
    log(f"shift {delta} of {n}, then a {L}-token entry: max|dlogit| {err:.2e}, oracle gap {s_ref.gap:.3f}")
    assert err <= TOL
    if s_ref.gap > 0.1:
        assert spp.ready_summary(r).argmax == s_ref.argmax
    for l in range(BF16.n_layers):
        K, V = read_kv(b, sess, l, n - delta + L)
        Ko, Vo = kv.layer(l)
        assert np.allclose(K, Ko[:, :n - delta + L], atol=4e-2, rtol=2.0 ** -7)
        assert np.allclose(V, Vo[:, :n - delta + L], atol=4e-2, rtol=2.0 ** -7)


def test_shift_invalidates_the_handle_and_rejects_bad_lengths():
    import torch
    import paper_2606_29565_amd as spp
    b = build_model(BF16, SEED, max_tokens=32)
    sess = spp.Session(b.model, 96)
    sess.append_delta(synth.cpu_tokens(40, SEED, 0, BF16.vocab).tolist())
    dist = torch.empty(BF16.vocab, dtype=torch.float32, device="cuda")
    r = sess.preposition([3, 4, 5], dist)
    spp.ready_summary(r)
    torch.cuda.synchronize()
    before = sess.kv.clone()
    info0 = sess.info()
    for bad in (0, -1, 41):
        with pytest.raises(spp.SppError):
            sess.shift(bad)
    torch.cuda.synchronize()
    assert torch.equal(sess.kv, before)
    info1 = sess.info()
    assert (info1.n_committed, info1.epoch, info1.valid) == (info0.n_committed, info0.epoch, info0.valid)
    sess.shift(40)  # everything dropped
    assert sess.info().n_committed == 0
    assert spp.gate(r, 0.0, None)[0] == spp.SPP_FALL_INVALID


def test_shift_at_the_8b_shape_on_sampled_cells():
    """One layer of the 8B shape, 8192 resident cells shifted by 1000: sampled cells of
    every kv head against the oracle's turn of the same synthetic cells."""
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.M8B.with_layers(1)
    n, delta = 8192, 1000
    b = build_model(shape, 5, max_tokens=32)
    sess = spp.Session(b.model, n + 64)
    fill_synthetic_kv(b, sess, 0, n)
    sess.restore(n)
    sess.shift(delta)
    torch.cuda.synchronize()
    K, V = read_kv(b, sess, 0, n - delta)
    rng = np.random.default_rng(0)
    cells = np.unique(np.concatenate([[0, 63, 64, 255, 256, n - delta - 1],
                                      rng.integers(0, n - delta, 200)]))
    for c in range(shape.n_kv):
        src_k = synth.kv_cpu(shape, 5, 0, 0, 0, c, n)[cells + delta]
        src_v = synth.kv_cpu(shape, 5, 0, 0, 1, c, n)[cells + delta]
        # every sampled cell turned at the one position -delta (rows of a single token)
        want = oracle.rope(src_k[None, :, :].astype(np.float64), -delta, shape.rope_base)[0]
        want = np.vectorize(oracle.round_bf16)(want)
        np.testing.assert_array_equal(V[c, cells], src_v)
        assert _key_close(K[c, cells], want, True), max_abs(K[c, cells], want)
    log(f"8B shape: {n} cells shifted by {delta}, {len(cells)} sampled cells x {shape.n_kv} heads match")
