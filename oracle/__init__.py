"""CPU oracle for the pre-position step and the confidence gate (fp64).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2606_29565_amd``) never imports, links or calls it, and shares no code
with it: the only common dependency is the seeded input generator in ``synth``.

Every function follows a passage of the paper:
  * ``forward``: the pre-position step of Alg. 1 (Sec. 3.2): append the entry at
    the live end n_s, one forward pass over the entry tokens only against the
    resident cells, ready distribution = logits at the decision point
    p = n_s + L_entry (Eq. (decision-point), Sec. 2.1).  The decoder layers are
    the standard ones of the workloads (the paper does not describe the model).
  * ``summary``: top-2 and gap gamma = l(1) - l(2) (Eq. (gap)), argmax, and the
    log-sum-exp of the distribution.
  * ``gate``: Alg. 2 with the gate of Eq. (gate), strict gamma > tau.
  * ``SessionModel``: the session state machine of Fig. "state" and Sec. 3.6.
  * ``dequant_mxfp4``: the 4-bit weights of the 70B-class headline model (Sec. 4 measures
    it at 4-bit precision without naming the format; the reading taken here is MXFP4,
    the OCP microscaling format): w = 2^(E - 127) * e2m1(code), one 8-bit scale byte E
    per 32 consecutive weights of a row.

Pins: tests/test_oracle_pins.py (values fixed by mathematics, library routines,
brute force and invariants) and tests/golden/ (tables written from the paper).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")

SERVED, FALL_INVALID, FALL_INELIGIBLE, FALL_GAP, FALL_NOT_IN_SET, FALL_NONFINITE = range(6)
OUTCOME_NAMES = ["SERVED", "FALL_INVALID", "FALL_INELIGIBLE", "FALL_GAP", "FALL_NOT_IN_SET",
                 "FALL_NONFINITE"]


def build(verbose: bool = False) -> None:
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", LIB,
           os.path.join(HERE, "oracle.c"), "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


class _Shape(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_q", ctypes.c_int32), ("n_kv", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("eps", ctypes.c_double), ("rope_base", ctypes.c_double),
                ("cache_bf16", ctypes.c_int32)]


class _LayerW(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")]


class _Summary(ctypes.Structure):
    _fields_ = [("argmax", ctypes.c_int32), ("second", ctypes.c_int32),
                ("top1", ctypes.c_double), ("top2", ctypes.c_double), ("gap", ctypes.c_double),
                ("lse", ctypes.c_double), ("nonfinite", ctypes.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"{LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.orc_rmsnorm.argtypes = [i32, i32, P, P, f64, P]
        L.orc_linear.argtypes = [i32, i32, i32, P, P, P]
        L.orc_rope.argtypes = [i32, i32, i32, P, i64, f64]
        L.orc_attention.argtypes = [i32, i32, i32, i32, P, P, P, i64, i64, P]
        L.orc_swiglu.argtypes = [i32, i32, P, P, P]
        L.orc_round_bf16.argtypes = [f64]
        L.orc_round_bf16.restype = f64
        L.orc_embed.argtypes = [i32, i32, P, P, P]
        L.orc_layer.argtypes = [P, P, P, P, i64, i64, i32, P]
        L.orc_layer.restype = ctypes.c_int
        L.orc_layer_last.argtypes = [P, P, P, P, i64, i64, i32, P]
        L.orc_layer_last.restype = ctypes.c_int
        L.orc_logits.argtypes = [P, P, P, P, P, P]
        L.orc_summary_of.argtypes = [i32, P, P]
        L.orc_shift_cells.argtypes = [i32, i64, i32, P, P, i64, i64, f64, i32]
        L.orc_shift_cells.restype = ctypes.c_int
        L.orc_gate.argtypes = [i32, i32, i32, f64, f64, i32]
        L.orc_gate.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


# ---------------------------------------------------------------------------------------
# pieces (thin wrappers, used by the pins)


def rmsnorm(x, g, eps: float) -> np.ndarray:
    x = _f64(np.atleast_2d(x)); g = _f32(g)
    out = np.empty_like(x)
    lib().orc_rmsnorm(x.shape[0], x.shape[1], _p(x), _p(g), eps, _p(out))
    return out


def linear(x, W) -> np.ndarray:
    x = _f64(np.atleast_2d(x)); W = _f32(W)
    assert W.shape[1] == x.shape[1]
    y = np.empty((x.shape[0], W.shape[0]), dtype=np.float64)
    lib().orc_linear(x.shape[0], W.shape[0], x.shape[1], _p(x), _p(W), _p(y))
    return y


def rope(u, pos0: int, base: float) -> np.ndarray:
    """u: [M, H, dh]; returns a rotated copy."""
    u = _f64(u).copy()
    M, H, dh = u.shape
    lib().orc_rope(M, H, dh, _p(u), pos0, base)
    return u


def attention(q, Kc, Vc, n_past: int) -> np.ndarray:
    """q: [M, Hq, dh] fp64; Kc, Vc: [Hkv, cap, dh] (cached cells)."""
    q = _f64(q); Kc = _f32(Kc); Vc = _f32(Vc)
    M, Hq, dh = q.shape
    Hkv, cap, _ = Kc.shape
    out = np.empty_like(q)
    lib().orc_attention(M, Hq, Hkv, dh, _p(q), _p(Kc), _p(Vc), cap, n_past, _p(out))
    return out


def swiglu(gate, up) -> np.ndarray:
    gate = _f64(np.atleast_2d(gate)); up = _f64(np.atleast_2d(up))
    out = np.empty_like(gate)
    lib().orc_swiglu(gate.shape[0], gate.shape[1], _p(gate), _p(up), _p(out))
    return out


def shift_cells(shape: synth.Shape, kv: "KVState", n_s: int, delta: int) -> None:
    """Sliding-window shift of every layer's cells in `kv` (Sec. 3.6): cells [delta, n_s)
    move to [0, n_s - delta), keys turned back by delta positions, values unchanged."""
    L = lib()
    for l in range(shape.n_layers):
        K, V = kv.layer(l)
        rc = L.orc_shift_cells(shape.n_kv, kv.cap, shape.head_dim, _p(K), _p(V), n_s, delta,
                               shape.rope_base, 1 if shape.bf16 else 0)
        if rc != 0:
            raise ValueError("orc_shift_cells rejected its arguments")


def round_bf16(v: float) -> float:
    return lib().orc_round_bf16(float(v))


# ---------------------------------------------------------------------------------------
# 4-bit weights (MXFP4)


def e2m1_value(code: int) -> float:
    """Value of a 4-bit e2m1 code (OCP microscaling formats): bit 3 sign, bits 2..1
    exponent e (bias 1), bit 0 mantissa m; e = 0 is subnormal, 0.5 * m, else
    2^(e - 1) * (1 + m / 2).  No infinities or NaNs."""
    sign = -1.0 if code & 8 else 1.0
    e, m = (code >> 1) & 3, code & 1
    mag = 0.5 * m if e == 0 else 2.0 ** (e - 1) * (1.0 + 0.5 * m)
    return sign * mag


def dequant_mxfp4(codes, scales) -> np.ndarray:
    """float32 weights [rows][cols] of one MXFP4 matrix: codes uint8 [rows][cols/2] (two
    codes per byte, the even column in the low nibble), scale bytes uint8 [rows][cols/32]:
    w[r][c] = 2^(scales[r][c // 32] - 127) * e2m1(code[r][c]).  Every value is exact in
    float32 (a 2-bit significand times a power of two)."""
    codes = np.asarray(codes, dtype=np.uint8)
    scales = np.asarray(scales, dtype=np.uint8)
    rows, half = codes.shape
    cols = 2 * half
    assert scales.shape == (rows, cols // 32)
    # float32 throughout: the table values, the powers of two and their products are exact
    table = np.array([e2m1_value(c) for c in range(16)], dtype=np.float32)
    q = np.empty((rows, cols), dtype=np.uint8)
    q[:, 0::2] = codes & 0x0F
    q[:, 1::2] = codes >> 4
    block_scale = np.ldexp(np.float32(1.0), scales.astype(np.int32) - 127)   # [rows][cols/32]
    w = table[q]
    w.reshape(rows, cols // 32, 32)[...] *= block_scale[:, :, None]
    return w


# ---------------------------------------------------------------------------------------
# model state


def _cshape(shape: synth.Shape) -> _Shape:
    return _Shape(shape.d_model, shape.n_q, shape.n_kv, shape.head_dim, shape.ffn, shape.vocab,
                  shape.eps, shape.rope_base, 1 if shape.bf16 else 0)


class Weights:
    """Weight provider: synthetic weights regenerated per layer unless cached."""

    def __init__(self, shape: synth.Shape, seed: int, lm_bias: Optional[np.ndarray] = None,
                 cache_layers: bool = True):
        self.shape, self.seed = shape, seed
        self.bias = None if lm_bias is None else _f32(lm_bias)
        self.cache_layers = cache_layers
        self._layers: Dict[int, Dict[int, np.ndarray]] = {}
        self._lm: Optional[np.ndarray] = None
        self._gf: Optional[np.ndarray] = None

    def layer(self, l: int) -> Dict[int, np.ndarray]:
        if l in self._layers:
            return self._layers[l]
        if self.shape.mxfp4:
            w = {}
            for k in range(9):
                if k in (synth.ATTN_NORM, synth.MLP_NORM):
                    w[k] = synth.weight_cpu(self.shape, self.seed, l, k)
                else:
                    w[k] = dequant_mxfp4(*synth.mxfp4_cpu(self.shape, self.seed, l, k))
        else:
            w = {k: synth.weight_cpu(self.shape, self.seed, l, k) for k in range(9)}
        if self.cache_layers:
            self._layers[l] = w
        return w

    def embed_rows(self, tokens: Sequence[int]) -> np.ndarray:
        d = self.shape.d_model
        return np.stack([synth.cpu_values(d, self.seed, synth.EMBED, synth.WEIGHT_SIGMA, 0.0,
                                          self.shape.bf16, lbase=int(t) * d) for t in tokens])

    def lm_head(self) -> np.ndarray:
        if self._lm is None:
            self._lm = synth.global_cpu(self.shape, self.seed, synth.LM_HEAD)
        return self._lm

    def final_norm(self) -> np.ndarray:
        if self._gf is None:
            self._gf = synth.global_cpu(self.shape, self.seed, synth.FINAL_NORM)
        return self._gf


class KVState:
    """Per-layer cached cells [n_kv, cap, head_dim] as float32 of the stored values.
    Layers materialise lazily; synthetic cells (N(0,1) draws) fill [0, n_synth)."""

    def __init__(self, shape: synth.Shape, cap: int, seed: int = 0, session: int = 0,
                 n_synth: int = 0):
        self.shape, self.cap = shape, cap
        self.seed, self.session, self.n_synth = seed, session, n_synth
        self._k: Dict[int, np.ndarray] = {}
        self._v: Dict[int, np.ndarray] = {}

    def layer(self, l: int) -> Tuple[np.ndarray, np.ndarray]:
        if l not in self._k:
            s = self.shape
            K = np.zeros((s.n_kv, self.cap, s.head_dim), dtype=np.float32)
            V = np.zeros_like(K)
            for c in range(s.n_kv):
                if self.n_synth:
                    K[c, :self.n_synth] = synth.kv_cpu(s, self.seed, self.session, l, 0, c, self.n_synth)
                    V[c, :self.n_synth] = synth.kv_cpu(s, self.seed, self.session, l, 1, c, self.n_synth)
            self._k[l], self._v[l] = K, V
        return self._k[l], self._v[l]

    def drop(self, l: int) -> None:
        self._k.pop(l, None)
        self._v.pop(l, None)


def forward(w: Weights, kv: KVState, n_past: int, tokens: Sequence[int],
            logits: bool = True, drop_layers: bool = False,
            hidden_out: Optional[List[np.ndarray]] = None,
            last_only: bool = False) -> Optional[np.ndarray]:
    """Append `tokens` at positions n_past.. and run them through the decoder.

    Returns the fp64 logits of the last token (the ready distribution when the
    tokens are an entry), or None when logits=False (a committed delta).
    `hidden_out`, when given, receives the residual stream after each layer.
    `last_only` computes the final layer for the last row only (its K/V cells for
    every row): the logits are unchanged, the other rows' final hidden states are not
    produced."""
    s = w.shape
    M = len(tokens)
    tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    x = np.ascontiguousarray(w.embed_rows(tok).astype(np.float64))
    cs = _cshape(s)
    for l in range(s.n_layers):
        lw = w.layer(l)
        K, V = kv.layer(l)
        arrs = [_f32(lw[k]) for k in range(9)]
        cw = _LayerW(*[a.ctypes.data for a in arrs])
        fn = lib().orc_layer_last if (last_only and l == s.n_layers - 1) else lib().orc_layer
        rc = fn(ctypes.byref(cs), ctypes.byref(cw), _p(K), _p(V), kv.cap, n_past, M, _p(x))
        if rc != 0:
            raise ValueError("orc_layer rejected its arguments")
        if hidden_out is not None:
            hidden_out.append(x.copy())
        if drop_layers:
            kv.drop(l)
    if not logits:
        return None
    out = np.empty(s.vocab, dtype=np.float64)
    last = np.ascontiguousarray(x[M - 1])
    lib().orc_logits(ctypes.byref(cs), _p(last), _p(_f32(w.final_norm())), _p(_f32(w.lm_head())),
                     _p(w.bias), _p(out))
    return out


@dataclasses.dataclass
class Summary:
    argmax: int
    second: int
    top1: float
    top2: float
    gap: float
    lse: float
    nonfinite: bool


def summary(logits) -> Summary:
    v = _f64(logits)
    s = _Summary()
    lib().orc_summary_of(v.shape[0], _p(v), ctypes.byref(s))
    return Summary(s.argmax, s.second, s.top1, s.top2, s.gap, s.lse, bool(s.nonfinite))


def gate(valid: bool, eligible: bool, nonfinite: bool, gap: float, tau: float,
         in_set: bool) -> int:
    return lib().orc_gate(int(valid), int(eligible), int(nonfinite), float(gap), float(tau),
                          int(in_set))


def in_bitmap(bitmap: np.ndarray, token: int) -> bool:
    return bool((int(bitmap[token >> 5]) >> (token & 31)) & 1)


# ---------------------------------------------------------------------------------------
# session state machine (Fig. "state", Sec. 3.2 and 3.6), host logic only


class SessionModel:
    """Reference session: committed tokens, speculative entry, ready record, epoch.

    * preposition (Alg. 1): skip when L_entry > B with B = capacity - used (no cell
      touched, valid <- false); else append the entry at n_s, valid <- true,
      position <- n_s + L_entry.
    * mutation (shift, rollback, update) clears valid in the same step and bumps
      the epoch (Sec. 3.6); an update first drops the speculative entry cells.
    * gate reads only (Alg. 2); the cached distribution serves repeated requests.
    * resume (Eq. (fallthrough), Sec. 3.5): a request that extends the entry by a delta
      keeps the entry cells in place (the constant-time restore), commits them with the
      delta, and one pass over the delta records a new ready distribution at the new
      end; with no entry present the delta is appended after the committed tokens.  It
      is the critical path, so it is bounded by the cells of the session, not by the
      idle-window budget.
    """

    def __init__(self, capacity: int, cells: Optional[int] = None):
        self.capacity = capacity             # idle-window budget B's bound
        self.cells = capacity if cells is None else cells
        self.committed: List[int] = []
        self.entry: List[int] = []
        self.valid = False
        self.epoch = 0
        self.position = -1

    @property
    def n_s(self) -> int:
        return len(self.committed)

    @property
    def used(self) -> int:
        return len(self.committed) + len(self.entry)

    def _invalidate(self) -> None:
        self.valid = False
        self.epoch += 1

    def preposition(self, entry: Sequence[int]) -> str:
        self.entry = []                      # a new pre-position replaces the old entry
        budget = self.capacity - self.n_s
        if len(entry) > budget:
            self.valid = False
            self.epoch += 1
            return "SKIPPED"
        self.entry = list(entry)
        self.epoch += 1
        self.valid = True
        self.position = self.n_s + len(entry)
        return "OK"

    def update(self, tokens: Sequence[int]) -> str:
        self.entry = []
        if self.n_s + len(tokens) > self.capacity:
            self._invalidate()
            return "CAPACITY"
        self.committed.extend(tokens)
        self._invalidate()
        return "OK"

    def resume(self, delta: Sequence[int]) -> str:
        if self.used + len(delta) > self.cells:
            return "CAPACITY"
        self.committed.extend(self.entry)
        self.committed.extend(delta)
        self.entry = []
        self.epoch += 1
        self.valid = True
        self.position = self.n_s
        return "OK"

    def rollback(self, n: int) -> None:
        self.entry = []
        self.committed = self.committed[:max(0, min(n, self.n_s))]
        self._invalidate()

    def shift(self, delta: int = 0) -> str:
        """Sec. 3.6 shift: delta = 0 is a shift done elsewhere (invalidation only); delta
        >= 1 drops the oldest delta committed tokens (their cells relocate)."""
        if delta < 0 or delta > self.n_s:
            return "INVALID"
        self.entry = []
        self.committed = self.committed[delta:]
        self._invalidate()
        return "OK"

    def gate_precheck(self, epoch: int, realized: Optional[Sequence[int]]) -> Optional[int]:
        """Outcome decided before any scan, or None when the scan must run."""
        if not self.valid or epoch != self.epoch:
            return FALL_INVALID
        if realized is not None and list(realized) != self.entry:
            return FALL_INELIGIBLE
        return None


# --------------------------------------------------------------------------------------
# Gate calibration (Sec. 2.4): Eqs. (coverage) and (risk) over measured decision points,
# and the threshold rule "the smallest tau with r(tau) <= r_max".


def wilson(k: int, n: int, z: float = 1.959964) -> Tuple[float, float]:
    """Wilson score interval for k successes in n trials (the interval the paper prints
    for its coverage and false-accept rate)."""
    if n == 0:
        return 0.0, 1.0
    p = k / n
    den = 1.0 + z * z / n
    mid = (p + z * z / (2 * n)) / den
    half = z / den * np.sqrt(p * (1 - p) / n + z * z / (4 * n * n))
    return max(0.0, mid - half), min(1.0, mid + half)


def calibrate(gaps, in_set, correct, r_max: float, taus=None):
    """Returns (tau_star, curve): curve rows (tau, served, wrong, coverage, risk) over the
    candidate thresholds in ascending order (the given ones, or 0 and every distinct gap
    >= 0); tau_star is the smallest candidate with something served and risk <= r_max,
    or inf.  Served means gap > tau and the argmax in the fast-answer set (Eq. (gate))."""
    gaps = [float(np.float32(g)) for g in gaps]
    if taus is None:
        cand = sorted({0.0} | {g for g in gaps if g >= 0.0})
    else:
        cand = sorted({float(np.float32(t)) for t in taus})
    curve, tau_star = [], float("inf")
    for tau in cand:
        served = [i for i, g in enumerate(gaps) if g > tau and in_set[i]]
        wrong = sum(1 for i in served if not correct[i])
        risk = wrong / len(served) if served else float("nan")
        curve.append((tau, len(served), wrong, len(served) / len(gaps), risk))
        if served and risk <= r_max and tau_star == float("inf"):
            tau_star = tau
    return tau_star, curve

