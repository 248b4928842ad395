"""Speculative pre-positioning on one MI355X: thin Python binding of libspp.so.

Every call marshals arguments into the C ABI declared in ``include/spp.h``; all
device work runs in the library's HIP kernels.  PyTorch only provides device
memory (tensors whose data pointers are handed to the library) and streams.
There is no fallback: if ``libspp.so`` is missing or no GPU is present, the calls
raise.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspp.so")

# spp_status
SPP_OK, SPP_SKIPPED_BUDGET, SPP_YIELDED = 0, 1, 2
SPP_E_INVALID_ARG, SPP_E_CAPACITY, SPP_E_HIP, SPP_E_STATE, SPP_E_NOMEM = -1, -2, -3, -4, -5
# spp_gate_outcome
SPP_SERVED, SPP_FALL_INVALID, SPP_FALL_INELIGIBLE, SPP_FALL_GAP, SPP_FALL_NOT_IN_SET, \
    SPP_FALL_NONFINITE = range(6)
OUTCOME_NAMES = ["SERVED", "FALL_INVALID", "FALL_INELIGIBLE", "FALL_GAP", "FALL_NOT_IN_SET",
                 "FALL_NONFINITE"]
# spp_mutation
SPP_MUT_SHIFT, SPP_MUT_ROLLBACK, SPP_MUT_UPDATE = 0, 1, 2
SPP_DTYPE_F32, SPP_DTYPE_BF16 = 0, 1
SPP_W_Q, SPP_W_K, SPP_W_V, SPP_W_O, SPP_W_GATE, SPP_W_UP, SPP_W_DOWN = range(7)
SPP_WFMT_DTYPE, SPP_WFMT_MXFP4 = 0, 1
# largest session capacity in cells per layer (spp.h)
SPP_MAX_CAPACITY = 16777216 - 64


class spp_model_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_double), ("dtype", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("max_sessions", ctypes.c_int32),
                ("weights_packed", ctypes.c_int32), ("weight_format", ctypes.c_int32)]


_PP = ctypes.POINTER(ctypes.c_void_p)


class spp_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("lm_bias", ctypes.c_void_p),
                ("attn_norm", _PP), ("wq", _PP), ("wk", _PP), ("wv", _PP), ("wo", _PP),
                ("mlp_norm", _PP), ("w_gate", _PP), ("w_up", _PP), ("w_down", _PP),
                ("scales", _PP * 7)]


class spp_session_config(ctypes.Structure):
    _fields_ = [("capacity", ctypes.c_int32), ("budget", ctypes.c_int32)]


class spp_kv_layout(ctypes.Structure):
    _fields_ = [("k_offset", ctypes.c_int64), ("v_offset", ctypes.c_int64),
                ("k_stride", ctypes.c_int64 * 3), ("v_stride", ctypes.c_int64 * 3),
                ("elem_bytes", ctypes.c_int32)]


class spp_ready_t(ctypes.Structure):
    _fields_ = [("session_id", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("epoch", ctypes.c_uint64)]


class spp_summary(ctypes.Structure):
    _fields_ = [("argmax", ctypes.c_int32), ("top1", ctypes.c_float), ("top2", ctypes.c_float),
                ("gap", ctypes.c_float), ("lse", ctypes.c_float), ("position", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


class spp_session_info(ctypes.Structure):
    _fields_ = [("n_committed", ctypes.c_int32), ("used_cells", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("budget", ctypes.c_int32),
                ("position", ctypes.c_int32), ("valid", ctypes.c_int32),
                ("decoded", ctypes.c_int32), ("entry_len", ctypes.c_int32),
                ("epoch", ctypes.c_uint64)]


class spp_gate_point(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("served", ctypes.c_int32), ("wrong", ctypes.c_int32),
                ("coverage", ctypes.c_double), ("coverage_lo", ctypes.c_double),
                ("coverage_hi", ctypes.c_double), ("risk", ctypes.c_double),
                ("risk_lo", ctypes.c_double), ("risk_hi", ctypes.c_double)]


EXPORTS = ["spp_model_create", "spp_model_destroy", "spp_session_kv_bytes", "spp_session_kv_layout",
           "spp_session_create", "spp_session_destroy", "spp_session_id", "spp_session_restore",
           "spp_kv_append_delta", "spp_preposition", "spp_ready_summary", "spp_gate",
           "spp_invalidate_on_mutation", "spp_session_info", "spp_session_info_get",
           "spp_preposition_batch",
           "spp_gate_batch", "spp_last_error", "spp_profile_preposition", "spp_kernel_class_name",
           "spp_copy_reference", "spp_pack_weight", "spp_pack_weight_mxfp4", "spp_resume",
           "spp_shift", "spp_gate_calibrate", "spp_preposition_idle", "spp_gate_batch_noalloc",
           "spp_profile_preposition_batch"]

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libspp.so (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, u32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t
    st = ctypes.c_int
    sig = {
        "spp_model_create": (st, [ctypes.POINTER(spp_model_config), ctypes.POINTER(spp_weights), ctypes.POINTER(P)]),
        "spp_model_destroy": (st, [P]),
        "spp_session_kv_bytes": (sz, [P, i32]),
        "spp_session_kv_layout": (st, [P, i32, i32, ctypes.POINTER(spp_kv_layout)]),
        "spp_session_create": (st, [P, ctypes.POINTER(spp_session_config), P, sz, ctypes.POINTER(P)]),
        "spp_session_destroy": (st, [P]),
        "spp_session_id": (i32, [P]),
        "spp_session_restore": (st, [P, i32]),
        "spp_kv_append_delta": (st, [P, P, i32, P]),
        "spp_preposition": (st, [P, P, i32, P, P, P, ctypes.POINTER(spp_ready_t)]),
        "spp_preposition_idle": (st, [P, P, i32, P, P, P, i32, P, ctypes.POINTER(spp_ready_t)]),
        "spp_resume": (st, [P, P, i32, P, P, P, ctypes.POINTER(spp_ready_t)]),
        "spp_ready_summary": (st, [spp_ready_t, ctypes.POINTER(spp_summary)]),
        "spp_gate": (st, [spp_ready_t, f32, P, P, i32, P, ctypes.POINTER(i32), ctypes.POINTER(st),
                          ctypes.POINTER(spp_summary)]),
        "spp_invalidate_on_mutation": (st, [P, st, i32]),
        "spp_shift": (st, [P, i32, P]),
        "spp_gate_calibrate": (st, [i32, P, P, P, ctypes.c_double, ctypes.c_double, i32, P,
                                    ctypes.POINTER(spp_gate_point), i32, ctypes.POINTER(i32),
                                    ctypes.POINTER(f32)]),
        "spp_session_info": (st, [P, ctypes.POINTER(spp_session_info)]),
        "spp_session_info_get": (st, [P, ctypes.POINTER(spp_session_info)]),
        "spp_preposition_batch": (st, [i32, P, P, P, P, P, P, P]),
        "spp_gate_batch": (st, [i32, P, P, P, P, P, P]),
        "spp_gate_batch_noalloc": (st, [i32, P, P, P, P, P, P]),
        "spp_last_error": (ctypes.c_char_p, []),
        "spp_profile_preposition": (i32, [P, P, i32, P, P, i32, P, P]),
        "spp_profile_preposition_batch": (i32, [i32, P, P, P, P, P, P, P, i32, P, P]),
        "spp_kernel_class_name": (ctypes.c_char_p, [i32]),
        "spp_copy_reference": (st, [P, P, sz, P]),
        "spp_pack_weight": (st, [ctypes.POINTER(spp_model_config), i32, P, P, P]),
        "spp_pack_weight_mxfp4": (st, [ctypes.POINTER(spp_model_config), i32, P, P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


class SppError(RuntimeError):
    def __init__(self, rc: int, where: str):
        super().__init__(f"{where} -> {rc}: {lib().spp_last_error().decode()}")
        self.rc = rc


class YieldFlag:
    """The host word an idle-window pre-position watches: set() when a request arrives."""

    def __init__(self):
        self._word = ctypes.c_uint32(0)

    @property
    def address(self) -> int:
        return ctypes.addressof(self._word)

    def set(self) -> None:
        self._word.value = 1

    def clear(self) -> None:
        self._word.value = 0

    def is_set(self) -> bool:
        return self._word.value != 0


def check(rc: int, where: str) -> int:
    if rc < 0:
        raise SppError(rc, where)
    return rc


def _ptr(t) -> int:
    """Device pointer of a tensor (or an int that already is one)."""
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _host_i32(tokens) -> Tuple[ctypes.Array, int]:
    vals = [int(t) for t in tokens]
    arr = (ctypes.c_int32 * max(1, len(vals)))(*vals)
    return arr, len(vals)


LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")
# projection keys in spp_weight_kind order (the MXFP4 scales are listed the same way)
PROJ_KEYS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def model_config(n_layers: int, d_model: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 ffn_dim: int, vocab: int, rope_base: float, bf16: bool, rms_eps: float = 1e-5,
                 max_tokens: int = 128, max_sessions: int = 1,
                 weights_packed: bool = False, mxfp4: bool = False) -> spp_model_config:
    return spp_model_config(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab,
                            rms_eps, rope_base, SPP_DTYPE_BF16 if bf16 else SPP_DTYPE_F32,
                            max_tokens, max_sessions, 1 if weights_packed else 0,
                            SPP_WFMT_MXFP4 if mxfp4 else SPP_WFMT_DTYPE)


def pack_weight_mxfp4(cfg: spp_model_config, which: int, codes_src, scales_src, codes_dst,
                      scales_dst, stream=None) -> None:
    """spp_pack_weight_mxfp4: row-major MXFP4 codes and scales into the tiled layout."""
    check(lib().spp_pack_weight_mxfp4(ctypes.byref(cfg), which, ctypes.c_void_p(_ptr(codes_src)),
                                      ctypes.c_void_p(_ptr(scales_src)),
                                      ctypes.c_void_p(_ptr(codes_dst)),
                                      ctypes.c_void_p(_ptr(scales_dst)),
                                      ctypes.c_void_p(_stream(stream))), "spp_pack_weight_mxfp4")


class Model:
    """A decoder whose weights live in caller-owned device memory.

    weights: dict with "embed", "final_norm", "lm_head", optional "lm_bias" (fp32), and
    per-layer lists under LAYER_KEYS, each entry a tensor or a device pointer.  With
    mxfp4=True the projection lists hold the 4-bit codes and "scales" maps each key of
    PROJ_KEYS to the per-layer e8m0 scales."""

    def __init__(self, n_layers: int, d_model: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 ffn_dim: int, vocab: int, rope_base: float, bf16: bool, weights: Dict,
                 rms_eps: float = 1e-5, max_tokens: int = 128, max_sessions: int = 1,
                 weights_packed: bool = False, mxfp4: bool = False):
        self.cfg = model_config(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab,
                                rope_base, bf16, rms_eps, max_tokens, max_sessions, weights_packed,
                                mxfp4)
        self.vocab = vocab
        self._keep = weights  # the library stores non-owning pointers
        arrays = {}
        for k in LAYER_KEYS:
            ptrs = [_ptr(t) for t in weights[k]]
            if len(ptrs) != n_layers:
                raise ValueError(f"{k}: {len(ptrs)} layers, expected {n_layers}")
            arrays[k] = (ctypes.c_void_p * n_layers)(*ptrs)
        scale_arrays = (_PP * 7)()
        if mxfp4:
            for i, k in enumerate(PROJ_KEYS):
                ptrs = [_ptr(t) for t in weights["scales"][k]]
                if len(ptrs) != n_layers:
                    raise ValueError(f"scales {k}: {len(ptrs)} layers, expected {n_layers}")
                arrays["scales_" + k] = (ctypes.c_void_p * n_layers)(*ptrs)
                scale_arrays[i] = ctypes.cast(arrays["scales_" + k], _PP)
        self._arrays = arrays
        w = spp_weights(_ptr(weights["embed"]), _ptr(weights["final_norm"]),
                        _ptr(weights["lm_head"]), _ptr(weights.get("lm_bias")),
                        *[ctypes.cast(arrays[k], _PP) for k in LAYER_KEYS], scale_arrays)
        h = ctypes.c_void_p()
        check(lib().spp_model_create(ctypes.byref(self.cfg), ctypes.byref(w), ctypes.byref(h)),
              "spp_model_create")
        self.handle = h

    def close(self) -> None:
        if self.handle:
            lib().spp_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def kv_bytes(self, capacity: int) -> int:
        return lib().spp_session_kv_bytes(self.handle, capacity)

    def kv_layout(self, capacity: int, layer: int) -> spp_kv_layout:
        out = spp_kv_layout()
        check(lib().spp_session_kv_layout(self.handle, capacity, layer, ctypes.byref(out)),
              "spp_session_kv_layout")
        return out

    def profile_preposition(self, session: "Session", entry: Sequence[int], dist, stream=None):
        """Per-kernel-class device time (us) and launch counts of one pre-position."""
        n = 32
        times = (ctypes.c_float * n)()
        counts = (ctypes.c_int32 * n)()
        arr, L = _host_i32(entry)
        k = lib().spp_profile_preposition(session.handle, arr, L, ctypes.c_void_p(_ptr(dist)),
                                          ctypes.c_void_p(_stream(stream)), n, times, counts)
        check(k, "spp_profile_preposition")
        return {lib().spp_kernel_class_name(i).decode(): (times[i], counts[i]) for i in range(k)}


@dataclasses.dataclass
class Ready:
    handle: spp_ready_t
    status: int


class Session:
    """A session over a caller-owned KV buffer (a uint8 torch tensor unless given)."""

    def __init__(self, model: Model, capacity: int, budget: int = 0, kv=None, device="cuda"):
        self.model = model
        nbytes = model.kv_bytes(capacity)
        if kv is None:
            import torch
            kv = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.kv = kv
        cfg = spp_session_config(capacity, budget)
        h = ctypes.c_void_p()
        check(lib().spp_session_create(model.handle, ctypes.byref(cfg), ctypes.c_void_p(_ptr(kv)),
                                       nbytes, ctypes.byref(h)), "spp_session_create")
        self.handle = h
        self.capacity = capacity

    def close(self) -> None:
        if self.handle:
            lib().spp_session_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def id(self) -> int:
        return lib().spp_session_id(self.handle)

    def restore(self, n_tokens: int) -> None:
        check(lib().spp_session_restore(self.handle, n_tokens), "spp_session_restore")

    def append_delta(self, tokens: Sequence[int], stream=None) -> int:
        arr, n = _host_i32(tokens)
        return check(lib().spp_kv_append_delta(self.handle, arr, n, ctypes.c_void_p(_stream(stream))),
                     "spp_kv_append_delta")

    def preposition(self, entry: Sequence[int], dist, default_bitmap=None, stream=None) -> Ready:
        arr, L = _host_i32(entry)
        r = spp_ready_t()
        rc = check(lib().spp_preposition(self.handle, arr, L, ctypes.c_void_p(_ptr(dist)),
                                         ctypes.c_void_p(_ptr(default_bitmap)),
                                         ctypes.c_void_p(_stream(stream)), ctypes.byref(r)),
                   "spp_preposition")
        return Ready(r, rc)

    def preposition_idle(self, entry: Sequence[int], dist, flag: "YieldFlag", chunk_layers: int = 1,
                         default_bitmap=None, stream=None) -> Ready:
        """Idle-window pre-position (spp_preposition_idle): blocks until done, or returns
        with status SPP_YIELDED soon after `flag` is set from another thread."""
        arr, L = _host_i32(entry)
        r = spp_ready_t()
        rc = check(lib().spp_preposition_idle(self.handle, arr, L, ctypes.c_void_p(_ptr(dist)),
                                              ctypes.c_void_p(_ptr(default_bitmap)),
                                              ctypes.c_void_p(flag.address), chunk_layers,
                                              ctypes.c_void_p(_stream(stream)), ctypes.byref(r)),
                   "spp_preposition_idle")
        return Ready(r, rc)

    def resume(self, delta: Sequence[int], dist, default_bitmap=None, stream=None) -> Ready:
        """Fall-through resume (spp_resume): keep the entry cells, process the delta only."""
        arr, n = _host_i32(delta)
        r = spp_ready_t()
        rc = check(lib().spp_resume(self.handle, arr, n, ctypes.c_void_p(_ptr(dist)),
                                    ctypes.c_void_p(_ptr(default_bitmap)),
                                    ctypes.c_void_p(_stream(stream)), ctypes.byref(r)),
                   "spp_resume")
        return Ready(r, rc)

    def invalidate(self, kind: int, arg: int = 0) -> None:
        check(lib().spp_invalidate_on_mutation(self.handle, kind, arg), "spp_invalidate_on_mutation")

    def shift(self, delta: int, stream=None) -> None:
        """Sliding-window shift by `delta` cells (spp_shift)."""
        check(lib().spp_shift(self.handle, delta, ctypes.c_void_p(_stream(stream))), "spp_shift")

    def info(self) -> spp_session_info:
        out = spp_session_info()
        check(lib().spp_session_info(self.handle, ctypes.byref(out)), "spp_session_info")
        return out


def ready_summary(ready: Ready) -> spp_summary:
    out = spp_summary()
    check(lib().spp_ready_summary(ready.handle, ctypes.byref(out)), "spp_ready_summary")
    return out


def gate(ready: Ready, tau: float, bitmap=None, realized: Optional[Sequence[int]] = None,
         stream=None) -> Tuple[int, int, spp_summary]:
    """Alg. 2: returns (outcome, token or -1, scan summary)."""
    tok = ctypes.c_int32(-1)
    outc = ctypes.c_int(0)
    summ = spp_summary()
    if realized is None:
        arr, n = None, 0
    else:
        arr, n = _host_i32(realized)
    check(lib().spp_gate(ready.handle, tau, ctypes.c_void_p(_ptr(bitmap)), arr, n,
                         ctypes.c_void_p(_stream(stream)), ctypes.byref(tok), ctypes.byref(outc),
                         ctypes.byref(summ)), "spp_gate")
    return outc.value, tok.value, summ


class GateCall:
    """spp_gate (or, with n > 1 handles, spp_gate_batch) with its arguments marshalled
    once, as a serving loop keeps them: each call() is the C call alone.  outcomes() and
    tokens() read the last call's results."""

    def __init__(self, readies: Sequence[Ready], taus: Sequence[float], bitmaps, stream=None,
                 noalloc: bool = False):
        n = len(readies)
        self.n = n
        self._st = ctypes.c_void_p(_stream(stream))
        if n == 1 and not noalloc:
            self._args = (readies[0].handle, ctypes.c_float(float(taus[0])),
                          ctypes.c_void_p(_ptr(bitmaps[0])), None, 0, self._st)
            self._tok = ctypes.c_int32(-1)
            self._out = ctypes.c_int(0)
            self._fn = lib().spp_gate
            self._tail = (ctypes.byref(self._tok), ctypes.byref(self._out), None)
        else:
            self._rs = (spp_ready_t * n)(*[r.handle for r in readies])
            self._ts = (ctypes.c_float * n)(*[float(t) for t in taus])
            self._bms = (ctypes.c_void_p * n)(*[_ptr(b) for b in bitmaps])
            self._toks = (ctypes.c_int32 * n)()
            self._outs = (ctypes.c_int * n)()
            self._fn = lib().spp_gate_batch_noalloc if noalloc else lib().spp_gate_batch
            self._args = (n, self._rs, self._ts, self._bms, self._st, self._toks, self._outs)
            self._tail = ()

    def __call__(self) -> int:
        rc = self._fn(*self._args, *self._tail)
        if rc < 0:
            raise SppError(rc, "gate")
        return rc

    def outcomes(self) -> List[Tuple[int, int]]:
        if self._tail:
            return [(self._out.value, self._tok.value)]
        return [(self._outs[i], self._toks[i]) for i in range(self.n)]


def _batch_args(sessions, entries, dists):
    n = len(sessions)
    hs = (ctypes.c_void_p * n)(*[s.handle.value for s in sessions])
    arrs = [_host_i32(e)[0] for e in entries]
    eps = (ctypes.c_void_p * n)(*[ctypes.cast(a, ctypes.c_void_p).value for a in arrs])
    lens = (ctypes.c_int32 * n)(*[len(e) for e in entries])
    dps = (ctypes.c_void_p * n)(*[_ptr(d) for d in dists])
    return n, hs, eps, lens, dps, arrs


def preposition_batch(sessions: Sequence[Session], entries: Sequence[Sequence[int]], dists,
                      stream=None) -> List[Ready]:
    n, hs, eps, lens, dps, _keep = _batch_args(sessions, entries, dists)
    readies = (spp_ready_t * n)()
    stats = (ctypes.c_int * n)()
    check(lib().spp_preposition_batch(n, hs, eps, lens, dps, ctypes.c_void_p(_stream(stream)),
                                      readies, stats), "spp_preposition_batch")
    return [Ready(readies[i], stats[i]) for i in range(n)]


def profile_preposition_batch(sessions: Sequence[Session], entries: Sequence[Sequence[int]],
                              dists, stream=None):
    """Per-kernel-class device time (us) and launch counts of one batched pre-position."""
    n, hs, eps, lens, dps, _keep = _batch_args(sessions, entries, dists)
    readies = (spp_ready_t * n)()
    stats = (ctypes.c_int * n)()
    nc = 32
    times = (ctypes.c_float * nc)()
    counts = (ctypes.c_int32 * nc)()
    k = lib().spp_profile_preposition_batch(n, hs, eps, lens, dps, ctypes.c_void_p(_stream(stream)),
                                            readies, stats, nc, times, counts)
    check(k, "spp_profile_preposition_batch")
    return {lib().spp_kernel_class_name(i).decode(): (times[i], counts[i]) for i in range(k)}


def gate_batch(readies: Sequence[Ready], taus: Sequence[float], bitmaps, stream=None,
               noalloc: bool = False):
    """spp_gate_batch (or, with noalloc, spp_gate_batch_noalloc): [(outcome, token)]."""
    n = len(readies)
    rs = (spp_ready_t * n)(*[r.handle for r in readies])
    ts = (ctypes.c_float * n)(*[float(t) for t in taus])
    bms = (ctypes.c_void_p * n)(*[_ptr(b) for b in bitmaps])
    toks = (ctypes.c_int32 * n)()
    outs = (ctypes.c_int * n)()
    name = "spp_gate_batch_noalloc" if noalloc else "spp_gate_batch"
    check(getattr(lib(), name)(n, rs, ts, bms, ctypes.c_void_p(_stream(stream)), toks, outs), name)
    return [(outs[i], toks[i]) for i in range(n)]


def pack_weight(cfg: spp_model_config, which: int, src, dst, stream=None) -> None:
    """Row-major projection weight `which` (SPP_W_*) of a model with configuration cfg ->
    the tiled layout spp_model_create expects with weights_packed (spp_pack_weight)."""
    check(lib().spp_pack_weight(ctypes.byref(cfg), which, ctypes.c_void_p(_ptr(src)),
                                ctypes.c_void_p(_ptr(dst)), ctypes.c_void_p(_stream(stream))),
          "spp_pack_weight")


def copy_reference(dst, src, nbytes: int, stream=None) -> None:
    check(lib().spp_copy_reference(ctypes.c_void_p(_ptr(dst)), ctypes.c_void_p(_ptr(src)), nbytes,
                                   ctypes.c_void_p(_stream(stream))), "spp_copy_reference")


def gate_calibrate(gaps, in_set, correct, r_max: float, taus=None, z: float = 1.959964):
    """spp_gate_calibrate: (tau_star, [spp_gate_point]) for the decision points' gaps,
    set membership and correctness (host arrays); tau_star is inf when no threshold keeps
    the risk within r_max."""
    import numpy as np
    g = np.ascontiguousarray(gaps, dtype=np.float32)
    a = np.ascontiguousarray(in_set, dtype=np.uint8)
    c = np.ascontiguousarray(correct, dtype=np.uint8)
    n = len(g)
    if len(a) != n or len(c) != n:
        raise ValueError("gaps, in_set and correct differ in length")
    t = None if taus is None else np.ascontiguousarray(taus, dtype=np.float32)
    cap = (len(t) if t is not None else n + 1)
    pts = (spp_gate_point * max(cap, 1))()
    npts, tau_star = ctypes.c_int32(), ctypes.c_float()
    check(lib().spp_gate_calibrate(n, ctypes.c_void_p(g.ctypes.data), ctypes.c_void_p(a.ctypes.data),
                                   ctypes.c_void_p(c.ctypes.data), float(r_max), float(z),
                                   0 if t is None else len(t),
                                   None if t is None else ctypes.c_void_p(t.ctypes.data), pts, cap,
                                   ctypes.byref(npts), ctypes.byref(tau_star)),
          "spp_gate_calibrate")
    return float(tau_star.value), [pts[i] for i in range(npts.value)]
