"""The fp16 range of the bf16 attention path.  bf16 models multiply attention in fp16:
every bf16 K/V cell of magnitude in [2^-14, 65504] is exact in fp16, smaller ones keep
fp16's absolute resolution (2^-24), and the query enters scaled by log2(e)/sqrt(dh) with
11 significant bits.  In-range extremes -- cells of magnitude 59904 and ~1e-7, a query
projection scaled so the scaled queries reach ~3e4 -- must still match the oracle.
Inputs beyond the range (a cell of 2^17, a scaled query above 65504) must flag the
distribution (summary flag bit 2) so that the gate never serves it, per session of a
batched pass."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import log, max_abs

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape("range", 2, 256, 4, 2, 64, 512, 2048, 1e4, "bf16")
SEED = 57
N_PAST, L = 100, 12


def _model(wq0_scale=1.0, max_sessions=1):
    import paper_2606_29565_amd as spp
    w = synth.gpu_weights(SHAPE, SEED)
    if wq0_scale != 1.0:
        w["wq"][0].mul_(wq0_scale)   # a power of two: exact in bf16, the oracle scales alike
    return spp.Model(SHAPE.n_layers, SHAPE.d_model, SHAPE.n_q, SHAPE.n_kv, SHAPE.head_dim,
                     SHAPE.ffn, SHAPE.vocab, SHAPE.rope_base, True, w, rms_eps=SHAPE.eps,
                     max_tokens=64, max_sessions=max_sessions)


def _session(model, session_id, plants):
    """A session with N_PAST synthetic cells and planted values: plants is a list of
    (layer, K or V, kv head, position, value) set over every dim of that cell."""
    import torch
    import paper_2606_29565_amd as spp
    sess = spp.Session(model, N_PAST + L)
    for l in range(SHAPE.n_layers):
        synth.gpu_fill_kv(sess.kv.data_ptr(), model.kv_layout(sess.capacity, l), SHAPE, SEED,
                          session_id, l, N_PAST)
    for (l, which, h, p, val) in plants:
        lay = model.kv_layout(sess.capacity, l)
        off, st = (lay.k_offset, lay.k_stride) if which == 0 else (lay.v_offset, lay.v_stride)
        el = sess.kv[off:].view(torch.bfloat16)
        for d in range(SHAPE.head_dim):
            sign = 1.0 if d % 3 else -1.0
            el[h * st[0] + p * st[1] + d * st[2]] = sign * val
    torch.cuda.synchronize()
    sess.restore(N_PAST)
    return sess


def _oracle(session_id, plants, wq0_scale=1.0):
    w = oracle.Weights(SHAPE, SEED, cache_layers=True)
    if wq0_scale != 1.0:
        w.layer(0)[synth.WQ] *= np.float32(wq0_scale)
    kv = oracle.KVState(SHAPE, N_PAST + L, seed=SEED, session=session_id, n_synth=N_PAST)
    for (l, which, h, p, val) in plants:
        arr = kv.layer(l)[which]
        for d in range(SHAPE.head_dim):
            arr[h, p, d] = (1.0 if d % 3 else -1.0) * np.float32(oracle.round_bf16(val))
    entry = synth.cpu_tokens(L, SEED, 3, SHAPE.vocab)
    return entry, oracle.forward(w, kv, N_PAST, entry)


IN_RANGE = [(0, 0, 1, 17, 59904.0), (0, 1, 0, 33, 59904.0), (1, 0, 1, 64, 59904.0),
            (1, 1, 1, 90, 59904.0), (0, 0, 0, 5, 1.0e-7), (0, 1, 1, 6, 1.0e-7),
            (1, 0, 0, 7, 1.5e-7)]


def test_in_range_extremes_match_the_oracle():
    import torch
    import paper_2606_29565_amd as spp
    scale = float(2 ** 17)   # scaled queries up to ~3e4 in layer 0
    model = _model(scale)
    sess = _session(model, 0, IN_RANGE)
    entry, ref = _oracle(0, IN_RANGE, scale)
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    r = sess.preposition(entry.tolist(), dist)
    summ = spp.ready_summary(r)
    got = dist.cpu().numpy()
    err = max_abs(got, ref)
    log(f"in-range extremes: max|dlogit| = {err:.3e}, flags {summ.flags}")
    assert err <= 5e-2
    assert summ.flags & 4 == 0
    out, _, _ = spp.gate(r, 0.0, None)
    assert out != spp.SPP_FALL_NONFINITE
    sess.close()
    model.close()


@pytest.mark.parametrize("case", ["cell", "query"])
def test_out_of_range_input_flags_and_never_serves(case):
    import torch
    import paper_2606_29565_amd as spp
    model = _model(float(2 ** 24) if case == "query" else 1.0)
    plants = [(1, 1, 1, 40, 131072.0)] if case == "cell" else []
    sess = _session(model, 0, plants)
    entry = synth.cpu_tokens(L, SEED, 3, SHAPE.vocab)
    dist = torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda")
    r = sess.preposition(entry.tolist(), dist)
    summ = spp.ready_summary(r)
    log(f"out of range ({case}): flags {summ.flags}")
    assert summ.flags & 4
    # (an overflowing input turns the scores and the logits to NaN here: no argmax to
    # put in the set, so every token is)
    bm = torch.from_numpy(synth.bitmap_from_ids(SHAPE.vocab, range(SHAPE.vocab))).cuda()
    out, tok, scan = spp.gate(r, 0.0, bm)
    assert out == spp.SPP_FALL_NONFINITE and tok == -1 and scan.flags & 4
    if case == "cell":
        # the range word belongs to the step: a clean session's next pre-position is clear
        # (in the query case every query of this model overflows)
        clean = _session(model, 1, [])
        r2 = clean.preposition(entry.tolist(), dist)
        assert spp.ready_summary(r2).flags & 4 == 0
        clean.close()
    sess.close()
    model.close()


def test_range_flag_is_per_session_in_a_batch():
    import torch
    import paper_2606_29565_amd as spp
    model = _model(1.0, max_sessions=4)
    plants = {1: [(0, 0, 0, 12, 131072.0)], 3: [(1, 1, 1, 3, 131072.0)]}
    sessions = [_session(model, i, plants.get(i, [])) for i in range(4)]
    entries = [synth.cpu_tokens(L - i, SEED, 10 + i, SHAPE.vocab).tolist() for i in range(4)]
    dists = [torch.empty(SHAPE.vocab, dtype=torch.float32, device="cuda") for _ in range(4)]
    readies = spp.preposition_batch(sessions, entries, dists)
    flags = [spp.ready_summary(r).flags & 4 for r in readies]
    assert [bool(f) for f in flags] == [False, True, False, True]
    res = spp.gate_batch(readies, [0.0] * 4, [None] * 4)
    assert [o == spp.SPP_FALL_NONFINITE for o, _ in res] == [False, True, False, True]
    for s in sessions:
        s.close()
    model.close()
