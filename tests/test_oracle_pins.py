"""Pins of the CPU oracle against things other than itself.

Each test checks an oracle function against a closed form, an independent library
routine the oracle does not use (numpy, torch, scipy), brute force, or an invariant the
method fixes, chosen so that a dropped term, a wrong sign or index, or a transposed
operand fails at least one of them.  CPU only.
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------------------- RMSNorm


def test_rmsnorm_closed_form():
    out = oracle.rmsnorm([[3.0, 4.0]], np.array([1.0, 1.0]), 0.0)
    r = math.sqrt((9 + 16) / 2)
    np.testing.assert_allclose(out[0], [3 / r, 4 / r], rtol=0, atol=1e-15)
    out = oracle.rmsnorm([[3.0, 4.0]], np.array([2.0, 0.5]), 0.0)
    np.testing.assert_allclose(out[0], [6 / r, 2 / r], rtol=0, atol=1e-15)
    # eps enters inside the root: x = [1, 1], eps = 3 -> 1/sqrt(1 + 3) = 0.5
    np.testing.assert_allclose(oracle.rmsnorm([[1.0, 1.0]], np.ones(2), 3.0)[0], [0.5, 0.5])


def test_rmsnorm_matches_torch_and_is_scale_invariant():
    x = RNG.standard_normal((5, 37))
    g = RNG.standard_normal(37).astype(np.float32)
    ours = oracle.rmsnorm(x, g, 1e-5)
    ref = F.rms_norm(torch.from_numpy(x), (37,), weight=torch.from_numpy(g.astype(np.float64)),
                     eps=1e-5).numpy()
    np.testing.assert_allclose(ours, ref, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.rmsnorm(7.5 * x, g, 0.0), oracle.rmsnorm(x, g, 0.0),
                               rtol=1e-13, atol=1e-13)
    unit = oracle.rmsnorm(x, np.ones(37, np.float32), 0.0)
    np.testing.assert_allclose((unit ** 2).mean(axis=1), 1.0, rtol=1e-13)


# ---------------------------------------------------------------------------- linear


def test_linear_matches_numpy_nonsquare():
    x = RNG.standard_normal((3, 7))
    W = RNG.standard_normal((5, 7)).astype(np.float32)
    np.testing.assert_allclose(oracle.linear(x, W), x @ W.astype(np.float64).T, rtol=1e-13,
                               atol=1e-13)
    eye = np.eye(7, dtype=np.float32)
    np.testing.assert_array_equal(oracle.linear(x, eye), x)


# ---------------------------------------------------------------------------- RoPE


def test_rope_is_identity_at_position_zero():
    u = RNG.standard_normal((1, 3, 8))
    np.testing.assert_array_equal(oracle.rope(u, 0, 1e4), u)


def test_rope_equals_complex_rotation():
    # pair (i, i + dh/2) is the complex number a + ib, rotated by e^{i P base^(-2i/dh)}
    dh, base, H = 8, 500.0, 2
    u = RNG.standard_normal((4, H, dh))
    pos0 = 37
    out = oracle.rope(u, pos0, base)
    half = dh // 2
    z = u[..., :half] + 1j * u[..., half:]
    P = (pos0 + np.arange(4))[:, None, None]
    freqs = base ** (-2.0 * np.arange(half) / dh)
    rz = z * np.exp(1j * P * freqs[None, None, :])
    np.testing.assert_allclose(out[..., :half], rz.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out[..., half:], rz.imag, rtol=0, atol=1e-12)


def test_rope_preserves_norm_and_depends_on_relative_position():
    dh, base = 16, 1e4
    q = RNG.standard_normal((1, 1, dh))
    k = RNG.standard_normal((1, 1, dh))
    qa = oracle.rope(q, 100, base)
    np.testing.assert_allclose(np.linalg.norm(qa), np.linalg.norm(q), rtol=1e-13)
    d1 = float((oracle.rope(q, 100, base) * oracle.rope(k, 40, base)).sum())
    d2 = float((oracle.rope(q, 1100, base) * oracle.rope(k, 1040, base)).sum())
    d3 = float((oracle.rope(q, 100, base) * oracle.rope(k, 41, base)).sum())
    assert abs(d1 - d2) < 1e-9
    assert abs(d1 - d3) > 1e-6


# ---------------------------------------------------------------------------- shift


def _shift_layer(n_kv, cap, dh, K, V, n_s, delta, base, bf16=False):
    import ctypes
    K = np.ascontiguousarray(K, dtype=np.float32)
    V = np.ascontiguousarray(V, dtype=np.float32)
    rc = oracle.lib().orc_shift_cells(n_kv, cap, dh, K.ctypes.data_as(ctypes.c_void_p),
                                      V.ctypes.data_as(ctypes.c_void_p), n_s, delta, base,
                                      1 if bf16 else 0)
    return rc, K, V


def test_shift_turns_cached_keys_to_their_new_positions():
    """A key cached at position p, moved to p - delta by the shift, equals the complex
    rotation of its unrotated vector at p - delta (Sec. 3.6 relocation with rotate-half
    RoPE: pair (i, i + dh/2) is a + ib turned by e^{i p base^(-2i/dh)}).  Values move
    unchanged; cells past the new end keep their contents."""
    n_kv, dh, base, n_s, cap, delta = 2, 16, 500.0, 11, 13, 4
    half = dh // 2
    k = RNG.standard_normal((n_kv, n_s, dh))
    freqs = base ** (-2.0 * np.arange(half) / dh)

    def rot(u, P):
        z = (u[..., :half] + 1j * u[..., half:]) * np.exp(1j * P[..., None] * freqs)
        return np.concatenate([z.real, z.imag], axis=-1)

    P = np.arange(n_s, dtype=np.float64)[None, :].repeat(n_kv, 0)
    K = np.zeros((n_kv, cap, dh)); K[:, :n_s] = rot(k, P)
    V = RNG.standard_normal((n_kv, cap, dh))
    rc, K2, V2 = _shift_layer(n_kv, cap, dh, K, V, n_s, delta, base)
    assert rc == 0
    n_new = n_s - delta
    want = rot(k[:, delta:], P[:, :n_new])                      # same vectors at p - delta
    np.testing.assert_allclose(K2[:, :n_new], want, rtol=0, atol=2e-6)   # fp32 cache rounding
    np.testing.assert_array_equal(V2[:, :n_new], V.astype(np.float32)[:, delta:n_s])
    np.testing.assert_array_equal(K2[:, n_new:], K.astype(np.float32)[:, n_new:])
    assert _shift_layer(n_kv, cap, dh, K, V, n_s, 0, base)[0] != 0        # delta >= 1
    assert _shift_layer(n_kv, cap, dh, K, V, n_s, n_s + 1, base)[0] != 0  # delta <= n_s


def test_shift_keeps_attention_over_the_surviving_cells():
    """Attention is a function of relative positions: a query at position P over the cells
    [delta, n) at their old positions equals, after the shift, the same query at
    P - delta over the moved cells [0, n - delta)."""
    n_kv, dh, base, n, delta = 1, 32, 1e4, 9, 3
    kpre = RNG.standard_normal((n, 1, dh))
    K = oracle.rope(kpre, 0, base)[:, 0, :][None]     # cached keys at positions 0..n-1
    V = RNG.standard_normal((1, n, dh))
    q = RNG.standard_normal((1, 1, dh))
    P = n + 5
    qa = oracle.rope(q, P, base)[0, 0]
    s = (K[0, delta:] @ qa) / math.sqrt(dh)
    a = np.exp(s - s.max()); a /= a.sum()
    want = a @ V[0, delta:]
    rc, K2, V2 = _shift_layer(n_kv, n, dh, K, V, n, delta, base)
    assert rc == 0
    qb = oracle.rope(q, P - delta, base)
    got = oracle.attention(qb, K2[:, :n - delta], V2[:, :n - delta], n_past=n - delta - 1)
    np.testing.assert_allclose(got[0, 0], want, rtol=0, atol=1e-6)


def test_shift_rounds_keys_to_bf16_cache():
    n_kv, dh, cap, n_s, delta = 2, 8, 6, 6, 2
    K = np.array([[[oracle.round_bf16(v) for v in row] for row in blk]
                  for blk in RNG.standard_normal((n_kv, cap, dh))], dtype=np.float32)
    V = np.array(K)
    rc, K2, _ = _shift_layer(n_kv, cap, dh, K, V, n_s, delta, 1e4, bf16=True)
    assert rc == 0
    flat = K2[:, :n_s - delta].ravel()
    assert all(oracle.round_bf16(float(v)) == float(v) for v in flat)


def test_session_model_shift_drops_oldest_committed_tokens():
    m = oracle.SessionModel(capacity=32)
    m.update(list(range(10)))
    assert m.preposition([100, 101]) == "OK" and m.valid
    e = m.epoch
    assert m.shift(3) == "OK"
    assert m.committed == list(range(3, 10)) and m.entry == [] and not m.valid and m.epoch == e + 1
    assert m.shift(8) == "INVALID" and m.committed == list(range(3, 10))
    assert m.shift(0) == "OK" and m.committed == list(range(3, 10))


# ---------------------------------------------------------------------------- attention


def test_attention_single_cell_returns_its_value():
    Kc = RNG.standard_normal((1, 4, 8)).astype(np.float32)
    Vc = RNG.standard_normal((1, 4, 8)).astype(np.float32)
    q = RNG.standard_normal((1, 2, 8))
    out = oracle.attention(q, Kc, Vc, n_past=0)
    for h in range(2):
        np.testing.assert_allclose(out[0, h], Vc[0, 0], rtol=0, atol=1e-7)


def test_attention_zero_query_is_mean_of_visible_values():
    Kc = RNG.standard_normal((2, 10, 4)).astype(np.float32)
    Vc = RNG.standard_normal((2, 10, 4)).astype(np.float32)
    q = np.zeros((3, 4, 4))
    out = oracle.attention(q, Kc, Vc, n_past=5)
    for m in range(3):
        for h in range(4):
            np.testing.assert_allclose(out[m, h], Vc[h // 2, :6 + m].astype(np.float64).mean(0),
                                       rtol=1e-12, atol=1e-12)


def test_attention_matches_torch_sdpa_gqa_causal():
    Hq, Hkv, dh, n_past, M, cap = 8, 2, 16, 11, 5, 20
    Kc = RNG.standard_normal((Hkv, cap, dh)).astype(np.float32)
    Vc = RNG.standard_normal((Hkv, cap, dh)).astype(np.float32)
    q = RNG.standard_normal((M, Hq, dh))
    ours = oracle.attention(q, Kc, Vc, n_past)
    T = n_past + M
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]                       # [1, Hq, M, dh]
    kt = torch.from_numpy(Kc[:, :T].astype(np.float64))[None]             # [1, Hkv, T, dh]
    vt = torch.from_numpy(Vc[:, :T].astype(np.float64))[None]
    mask = torch.arange(T)[None, :] <= (n_past + torch.arange(M))[:, None]
    ref = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, enable_gqa=True)
    np.testing.assert_allclose(ours, ref[0].permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-12)


def test_attention_row_ignores_later_cells():
    Kc = RNG.standard_normal((1, 12, 8)).astype(np.float32)
    Vc = RNG.standard_normal((1, 12, 8)).astype(np.float32)
    q = RNG.standard_normal((3, 1, 8))
    a = oracle.attention(q, Kc, Vc, n_past=8)
    Kc2, Vc2 = Kc.copy(), Vc.copy()
    Kc2[0, 10] += 5.0
    Vc2[0, 10] -= 3.0
    b = oracle.attention(q, Kc2, Vc2, n_past=8)
    np.testing.assert_array_equal(a[:2], b[:2])
    assert np.abs(a[2] - b[2]).max() > 1e-3


# ---------------------------------------------------------------------------- SwiGLU, bf16


def test_swiglu_matches_torch():
    g = RNG.standard_normal((4, 9)) * 4
    u = RNG.standard_normal((4, 9))
    ref = (F.silu(torch.from_numpy(g)) * torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(oracle.swiglu(g, u), ref, rtol=1e-14, atol=1e-14)
    assert oracle.swiglu([[0.0]], [[5.0]])[0, 0] == 0.0


def test_round_bf16_ties_and_torch():
    assert oracle.round_bf16(1 + 2 ** -8) == 1.0                    # tie -> even (down)
    assert oracle.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6         # tie -> even (up)
    assert oracle.round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7  # just above the tie
    assert oracle.round_bf16(-3.0) == -3.0
    x = (RNG.standard_normal(2000) * 10.0 ** RNG.integers(-6, 6, 2000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    ours = np.array([oracle.round_bf16(float(v)) for v in x])
    np.testing.assert_array_equal(ours, ref)


# ---------------------------------------------------------------------------- decoder

TINY2 = synth.Shape("pin", 2, 64, 4, 2, 16, 96, 97, 1.0e4, "f32")


def _torch_decoder(shape, w: "oracle.Weights", tokens):
    """The same decoder written with torch library ops in fp64 (rotary as complex multiply)."""
    d, Hq, Hkv, dh = shape.d_model, shape.n_q, shape.n_kv, shape.head_dim
    T = len(tokens)
    x = torch.from_numpy(w.embed_rows(tokens).astype(np.float64))
    pos = torch.arange(T, dtype=torch.float64)
    half = dh // 2
    freqs = shape.rope_base ** (-2.0 * torch.arange(half, dtype=torch.float64) / dh)
    rot = torch.polar(torch.ones(T, half, dtype=torch.float64), pos[:, None] * freqs[None])

    def rotary(t):  # t: [T, H, dh]
        z = torch.complex(t[..., :half], t[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    def cache_round(t):
        return t.to(torch.bfloat16).to(torch.float64) if shape.bf16 else t.float().double()

    t64 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    for l in range(shape.n_layers):
        lw = w.layer(l)
        h = F.rms_norm(x, (d,), weight=t64(lw[synth.ATTN_NORM]), eps=shape.eps)
        q = rotary(F.linear(h, t64(lw[synth.WQ])).view(T, Hq, dh))
        k = cache_round(rotary(F.linear(h, t64(lw[synth.WK])).view(T, Hkv, dh)))
        v = cache_round(F.linear(h, t64(lw[synth.WV])).view(T, Hkv, dh))
        o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                           v.transpose(0, 1)[None], is_causal=True,
                                           enable_gqa=True)[0].transpose(0, 1).reshape(T, -1)
        x = x + F.linear(o, t64(lw[synth.WO]))
        h2 = F.rms_norm(x, (d,), weight=t64(lw[synth.MLP_NORM]), eps=shape.eps)
        x = x + F.linear(F.silu(F.linear(h2, t64(lw[synth.WG]))) * F.linear(h2, t64(lw[synth.WU])),
                         t64(lw[synth.WD]))
    z = F.rms_norm(x[-1], (d,), weight=t64(w.final_norm()), eps=shape.eps)
    bias = None if w.bias is None else t64(w.bias)
    return F.linear(z, t64(w.lm_head()), bias).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decoder_matches_torch_composition(dtype):
    shape = TINY2.with_dtype(dtype)
    w = oracle.Weights(shape, seed=77)
    toks = synth.cpu_tokens(13, 77, 0, shape.vocab)
    kv = oracle.KVState(shape, cap=16)
    ours = oracle.forward(w, kv, 0, toks)
    ref = _torch_decoder(shape, w, toks.tolist())
    np.testing.assert_allclose(ours, ref, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decoder_with_lm_head_bias_matches_torch_composition(dtype):
    # The decisive-logit workloads add an fp32 bias vector to the LM head's output (one
    # planted token far above the rest).  torch's linear with its bias argument, in fp64,
    # against the oracle's LM head with the bias: the planted token must win, by the
    # planted margin, at its own index.
    shape = TINY2.with_dtype(dtype)
    planted, beta = 41, 25.0
    bias = (RNG.standard_normal(shape.vocab) * 0.5).astype(np.float32)
    bias[planted] = beta
    w = oracle.Weights(shape, seed=78, lm_bias=bias)
    toks = synth.cpu_tokens(11, 78, 0, shape.vocab)
    ours = oracle.forward(w, oracle.KVState(shape, cap=16), 0, toks)
    ref = _torch_decoder(shape, w, toks.tolist())
    np.testing.assert_allclose(ours, ref, rtol=1e-10, atol=1e-10)
    s = oracle.summary(ours)
    assert s.argmax == planted and s.gap > beta / 2
    w0 = oracle.Weights(shape, seed=78)
    plain = oracle.forward(w0, oracle.KVState(shape, cap=16), 0, toks)
    # the bias moves no logit but through its own entry
    np.testing.assert_allclose(ours - plain, bias.astype(np.float64), rtol=0, atol=1e-12)
    # and synth.lm_bias plants beta at the token given, zero elsewhere
    b = synth.lm_bias(shape, 3.0, 7)
    assert b.dtype == np.float32 and b[7] == 3.0 and np.count_nonzero(b) == 1


def test_delta_append_equals_full_prefill_bit_exact():
    # The ready distribution depends only on the token sequence up to p (Sec. 3.6):
    # committing a prefix and appending the entry must equal one pass over the whole.
    shape = synth.TINY
    w = oracle.Weights(shape, seed=5)
    toks = synth.cpu_tokens(40, 5, 1, shape.vocab)
    kv_a = oracle.KVState(shape, cap=48)
    assert oracle.forward(w, kv_a, 0, toks[:28], logits=False) is None
    delta = oracle.forward(w, kv_a, 28, toks[28:])
    kv_b = oracle.KVState(shape, cap=48)
    full = oracle.forward(w, kv_b, 0, toks)
    np.testing.assert_array_equal(delta, full)
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(kv_a.layer(l)[0], kv_b.layer(l)[0])
        np.testing.assert_array_equal(kv_a.layer(l)[1], kv_b.layer(l)[1])


def test_mha_equals_gqa_with_replicated_kv_heads():
    # grouping: q head h reads kv head h // G; replicating every kv head G times turns the
    # model into multi-head attention with the same output.
    Hq, Hkv, dh = 4, 2, 8
    Kc = RNG.standard_normal((Hkv, 6, dh)).astype(np.float32)
    Vc = RNG.standard_normal((Hkv, 6, dh)).astype(np.float32)
    q = RNG.standard_normal((2, Hq, dh))
    gqa = oracle.attention(q, Kc, Vc, n_past=4)
    mha = oracle.attention(q, np.repeat(Kc, 2, axis=0), np.repeat(Vc, 2, axis=0), n_past=4)
    np.testing.assert_array_equal(gqa, mha)


# ---------------------------------------------------------------------------- summary, gate


def _brute_top2(v):
    order = sorted(range(len(v)), key=lambda i: (math.isnan(v[i]), -v[i] if not math.isnan(v[i]) else 0, i))
    return order[0], order[1]


def test_summary_matches_sort_and_logsumexp():
    for trial in range(20):
        V = int(RNG.integers(2, 3000))
        v = RNG.standard_normal(V) * 3
        if trial % 3 == 0:                       # planted exact ties at the top
            j = RNG.choice(V, size=min(V, 3), replace=False)
            v[j] = v.max() + 1.0
        s = oracle.summary(v)
        a, b = _brute_top2(v.tolist())
        assert (s.argmax, s.second) == (a, b)
        assert s.top1 == v[a] and s.top2 == v[b] and s.gap == v[a] - v[b]
        assert not s.nonfinite
        assert abs(s.lse - scipy.special.logsumexp(v)) < 1e-10
        assert abs(np.exp(v - s.lse).sum() - 1.0) < 1e-12
        assert v.max() <= s.lse <= v.max() + math.log(V) + 1e-12


def test_summary_ties_and_nonfinite():
    s = oracle.summary([1.0, 5.0, 5.0, 2.0])
    assert (s.argmax, s.second, s.gap) == (1, 2, 0.0)
    s = oracle.summary([1.0, float("nan"), 3.0, 2.0])
    assert s.nonfinite and (s.argmax, s.second) == (2, 3) and math.isnan(s.lse)
    s = oracle.summary([1.0, float("inf"), 3.0])
    assert s.nonfinite and s.argmax == 1
    s = oracle.summary([0.0, 7.0])
    assert (s.argmax, s.second, s.gap) == (1, 0, 7.0)


def _read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_gate_truth_table_from_alg2():
    rows = _read_table("gate_truth_table.txt")
    assert len(rows) >= 20
    for valid, elig, nonfin, gap, tau, in_set, expected in rows:
        got = oracle.gate(valid == "1", elig == "1", nonfin == "1", float(gap), float(tau),
                          in_set == "1")
        assert oracle.OUTCOME_NAMES[got] == expected, (valid, elig, nonfin, gap, tau, in_set)


def test_coverage_is_monotone_in_tau():
    # c(tau) = Pr(gap > tau and argmax in A) is non-increasing in tau (Sec. 2.4).
    gaps = np.abs(RNG.standard_normal(500)) * 3
    in_set = RNG.random(500) < 0.7
    cov = []
    for tau in np.linspace(0, 6, 25):
        cov.append(np.mean([oracle.gate(True, True, False, g, tau, s) == oracle.SERVED
                            for g, s in zip(gaps, in_set)]))
    assert all(a >= b for a, b in zip(cov, cov[1:]))
    assert cov[0] == pytest.approx(np.mean(in_set & (gaps > 0)))


def test_session_state_machine_golden():
    rows = _read_table("state_machine.txt")
    sess = None
    for r in rows:
        op = r[0]
        if op == "capacity":
            sess = oracle.SessionModel(int(r[1]))
        elif op == "upd":
            sess.update(list(range(int(r[1]))))
        elif op == "pp":
            sess.preposition(list(range(int(r[1]))))
        elif op == "rb":
            sess.rollback(int(r[1]))
        elif op == "shift":
            sess.shift()
        elif op == "gate":
            assert sess.gate_precheck(sess.epoch, None) in (None, oracle.FALL_INVALID)
        elif op == "res":
            sess.resume(list(range(int(r[1]))))
        elif op == "expect":
            got = [sess.n_s, sess.used, int(sess.valid), sess.position]
            assert got == [int(x) for x in r[1:]], (got, r)
        elif op == "end":
            sess = None


def test_last_row_mode_equals_full_layer():
    # the final-layer shortcut computes the same last row and the same cells
    shape = synth.TINY.with_layers(2)
    w = oracle.Weights(shape, seed=9)
    toks = synth.cpu_tokens(20, 9, 3, shape.vocab)
    kv_a = oracle.KVState(shape, cap=24)
    kv_b = oracle.KVState(shape, cap=24)
    oracle.forward(w, kv_a, 0, toks[:6], logits=False)
    oracle.forward(w, kv_b, 0, toks[:6], logits=False)
    full = oracle.forward(w, kv_a, 6, toks[6:])
    fast = oracle.forward(w, kv_b, 6, toks[6:], last_only=True)
    np.testing.assert_array_equal(full, fast)
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(kv_a.layer(l)[0], kv_b.layer(l)[0])
        np.testing.assert_array_equal(kv_a.layer(l)[1], kv_b.layer(l)[1])


# ---------------------------------------------------------------------------------------
# 4-bit weights (MXFP4): the dequantization the oracle applies to the headline model's
# 4-bit projections (Sec. 4 measures a 70B-class model at 4-bit precision)

# e2m1 magnitudes as the OCP Microscaling Formats specification (v1.0, FP4 E2M1) lists
# them for codes 0..7; codes 8..15 are their negatives
OCP_E2M1 = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def test_e2m1_table_matches_the_ocp_listing():
    got = [oracle.e2m1_value(c) for c in range(16)]
    assert got[:8] == OCP_E2M1
    assert got[8:] == [-v for v in OCP_E2M1]
    assert math.copysign(1.0, got[8]) == -1.0   # code 8 is negative zero


def test_dequant_mxfp4_hand_example():
    # one row of 64 weights: block 0 holds codes 0..15 twice with scale byte 127 (x1),
    # block 1 holds code 7 (6.0) and code 9 (-0.5) alternately with scale byte 130 (x8)
    codes = np.zeros((1, 32), dtype=np.uint8)
    for j in range(16):                      # elements 2j, 2j+1 of block 0
        lo, hi = (2 * j) % 16, (2 * j + 1) % 16
        codes[0, j] = lo | (hi << 4)
    codes[0, 16:] = 7 | (9 << 4)
    scales = np.array([[127, 130]], dtype=np.uint8)
    w = oracle.dequant_mxfp4(codes, scales)
    expect0 = OCP_E2M1 + [-v for v in OCP_E2M1]
    assert w.dtype == np.float32 and w.shape == (1, 64)
    assert w[0, :16].tolist() == expect0 and w[0, 16:32].tolist() == expect0
    assert w[0, 32:].tolist() == [48.0, -4.0] * 16


def test_dequant_mxfp4_scale_byte_doubles_only_its_block():
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 256, size=(3, 64), dtype=np.uint8)
    scales = rng.integers(110, 130, size=(3, 4), dtype=np.uint8)
    w = oracle.dequant_mxfp4(codes, scales)
    s2 = scales.copy()
    s2[1, 2] += 1
    w2 = oracle.dequant_mxfp4(codes, s2)
    assert np.array_equal(w2[1, 64:96], 2 * w[1, 64:96])
    mask = np.ones_like(w, dtype=bool)
    mask[1, 64:96] = False
    assert np.array_equal(w2[mask], w[mask])


def test_dequant_mxfp4_nibble_order_and_generator_bytes():
    # the even column is the low nibble: swapping the nibbles of one byte swaps two weights
    codes = np.array([[0x21] + [0] * 15], dtype=np.uint8)
    w = oracle.dequant_mxfp4(codes, np.array([[127]], dtype=np.uint8))
    assert w[0, 0] == 0.5 and w[0, 1] == 1.0
    # generated model bytes: every code value occurs, scale bytes stay in {119, 120, 121}
    shape = synth.Shape("q", 1, 128, 2, 2, 64, 128, 64, 1e4, "bf16", wfmt="mxfp4")
    c, s = synth.mxfp4_cpu(shape, 9, 0, synth.WQ)
    assert c.shape == (128, 64) and s.shape == (128, 4)
    assert set(np.unique(s).tolist()) <= {119, 120, 121}
    assert len(set((c & 15).ravel().tolist()) | set((c >> 4).ravel().tolist())) == 16
    # and a sub-range of the generator is the same bytes as the whole
    assert np.array_equal(synth.cpu_fp4_bytes(10, 9, synth.fp4_code_tid(0, synth.WQ), lbase=7),
                          c.ravel()[7:17])
