"""Seeded synthetic inputs: the only module both the oracle side and the HIP side use.

It holds no arithmetic of the method, only
  * the model shapes and workloads the tests and the bench run on,
  * a tensor-id scheme so that every weight, KV cell and token id is addressed by
    (seed, tensor id, logical index) alone, and
  * two independent implementations of the generator defined in ``synth.h``:
    a C one for the CPU (``libsynth_cpu.so``) and a HIP one for the GPU
    (``libsynth_gpu.so``).  A GPU test checks that they agree bit for bit.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
CPU_LIB = os.path.join(HERE, "libsynth_cpu.so")
GPU_LIB = os.path.join(HERE, "libsynth_gpu.so")

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose: bool = False) -> None:
    """Compile both generator libraries in place (always recompiles)."""
    cmds = [
        ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", CPU_LIB,
         os.path.join(HERE, "synth_cpu.c")],
        ["hipcc", *HIP_FLAGS, "-o", GPU_LIB, os.path.join(HERE, "synth_gpu.hip")],
    ]
    for c in cmds:
        if verbose:
            print(" ".join(c), flush=True)
        subprocess.run(c, check=True)


# ----------------------------------------------------------------------------------------
# tensor ids

ATTN_NORM, WQ, WK, WV, WO, MLP_NORM, WG, WU, WD = range(9)
EMBED, FINAL_NORM, LM_HEAD = 1, 2, 3
WEIGHT_SIGMA = 0.02
NORM_SIGMA = 0.02
KV_SIGMA = 1.0
POS_BITS = 24  # logical KV index = ((head << POS_BITS) | position) * head_dim + dim


def layer_tid(layer: int, kind: int) -> int:
    return ((layer + 1) << 8) | kind


def kv_tid(session: int, layer: int, which: int) -> int:
    """which: 0 = K, 1 = V."""
    return (1 << 40) | (session << 20) | (layer << 1) | which


def token_tid(stream: int) -> int:
    return (2 << 40) | stream


def fp4_code_tid(layer: int, kind: int) -> int:
    """4-bit codes of a projection of a model stored as MXFP4."""
    return (1 << 20) | layer_tid(layer, kind)


def fp4_scale_tid(layer: int, kind: int) -> int:
    """Block scale bytes of a projection of a model stored as MXFP4."""
    return (2 << 20) | layer_tid(layer, kind)


# ----------------------------------------------------------------------------------------
# shapes and workloads


@dataclasses.dataclass(frozen=True)
class Shape:
    name: str
    n_layers: int
    d_model: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int
    vocab: int
    rope_base: float
    dtype: str  # "f32" or "bf16": weights, KV cells and matrix-core operands
    eps: float = 1e-5
    wfmt: str = "dtype"  # projection storage: "dtype" or "mxfp4" (4-bit codes + scales)

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    @property
    def bf16(self) -> bool:
        return self.dtype == "bf16"

    def with_layers(self, n: int) -> "Shape":
        return dataclasses.replace(self, n_layers=n, name=f"{self.name}-L{n}")

    def with_dtype(self, dtype: str) -> "Shape":
        return dataclasses.replace(self, dtype=dtype, name=f"{self.name}-{dtype}")

    @property
    def mxfp4(self) -> bool:
        return self.wfmt == "mxfp4"

    def weight_numel(self) -> dict:
        d, q, kv, f = self.d_model, self.n_q * self.head_dim, self.n_kv * self.head_dim, self.ffn
        return {ATTN_NORM: d, WQ: q * d, WK: kv * d, WV: kv * d, WO: d * q,
                MLP_NORM: d, WG: f * d, WU: f * d, WD: d * f}

    def weight_shape(self, kind: int):
        d, q, kv, f = self.d_model, self.n_q * self.head_dim, self.n_kv * self.head_dim, self.ffn
        return {ATTN_NORM: (d,), WQ: (q, d), WK: (kv, d), WV: (kv, d), WO: (d, q),
                MLP_NORM: (d,), WG: (f, d), WU: (f, d), WD: (d, f)}[kind]

    def bytes_per_weight(self) -> int:
        return 2 if self.bf16 else 4


# The five workloads of the method's evaluation, as synthetic stand-ins (shapes only;
# the paper's own task data and trained models are not used).
TINY = Shape("tiny", 2, 256, 4, 4, 64, 1024, 4096, 1.0e4, "f32")
M8B = Shape("8b", 32, 4096, 32, 8, 128, 14336, 128256, 5.0e5, "bf16")
M32B = Shape("32b", 64, 5120, 64, 8, 128, 27648, 152064, 1.0e6, "bf16")
# the 70B-class headline model of the paper's measurements, stored at 4 bits (MXFP4)
M70B_FP4 = Shape("70b-mxfp4", 80, 8192, 64, 8, 128, 28672, 128256, 5.0e5, "bf16", wfmt="mxfp4")


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: Shape
    n_past: int            # persistent KV tokens n_s
    entry_len: int         # L_entry
    fast_set_size: int
    seed: int
    synthetic_kv: bool     # True: KV cells are N(0,1) draws; False: a real prefill
    lm_bias: float = 0.0   # planted logit bias beta on one token


WORKLOADS = {
    "tiny": Workload("tiny", TINY, 512, 16, 32, 1001, False, 0.0),
    "stream8b": Workload("stream8b", M8B, 8192, 32, 64, 1002, True, 0.0),
    "agentic8b": Workload("agentic8b", M8B, 32768, 128, 64, 1003, True, 0.0),
    "target32b": Workload("target32b", M32B, 16384, 32, 64, 1004, True, 10.1),
    "stream70b_mxfp4": Workload("stream70b_mxfp4", M70B_FP4, 8192, 32, 64, 1005, True, 0.0),
    # 64 sessions of the 8B model; resident cells and entry lengths per session from
    # batched_spec (n_past / entry_len here are the ranges' upper ends)
    "batched8b": Workload("batched8b", M8B, 8192, 64, 64, 1006, True, 0.0),
}


# ----------------------------------------------------------------------------------------
# CPU generator

_cpu = None
_gpu = None


def cpu_lib():
    global _cpu
    if _cpu is None:
        if not os.path.exists(CPU_LIB):
            raise RuntimeError(f"{CPU_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(CPU_LIB)
        lib.synth_fill_f32.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_uint64, ctypes.c_int64, ctypes.c_double,
                                       ctypes.c_float, ctypes.c_int]
        lib.synth_fill_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                        ctypes.c_uint64, ctypes.c_int64, ctypes.c_double,
                                        ctypes.c_float]
        lib.synth_fill_tokens.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                          ctypes.c_uint64, ctypes.c_int64, ctypes.c_uint32]
        lib.synth_fill_fp4.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_uint64, ctypes.c_int64]
        lib.synth_fill_e8m0.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                        ctypes.c_uint64, ctypes.c_int64]
        lib.synth_raw.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.synth_raw.restype = ctypes.c_uint64
        lib.synth_tensor_key.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.synth_tensor_key.restype = ctypes.c_uint64
        _cpu = lib
    return _cpu


def cpu_values(n: int, seed: int, tid: int, sigma: float, offset: float = 0.0,
               bf16: bool = False, lbase: int = 0) -> np.ndarray:
    """float32 array: elements lbase .. lbase+n-1 of tensor `tid` (bf16-rounded if asked)."""
    out = np.empty(n, dtype=np.float32)
    cpu_lib().synth_fill_f32(out.ctypes.data, n, seed, tid, lbase, sigma, offset, int(bf16))
    return out


def cpu_bf16_bits(n: int, seed: int, tid: int, sigma: float, offset: float = 0.0,
                  lbase: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.uint16)
    cpu_lib().synth_fill_bf16(out.ctypes.data, n, seed, tid, lbase, sigma, offset)
    return out


def cpu_tokens(n: int, seed: int, stream: int, vocab: int, lbase: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    cpu_lib().synth_fill_tokens(out.ctypes.data, n, seed, token_tid(stream), lbase, vocab)
    return out


def cpu_fp4_bytes(nbytes: int, seed: int, tid: int, lbase: int = 0) -> np.ndarray:
    """uint8 code bytes lbase .. lbase+nbytes-1 (two 4-bit codes each, even one low)."""
    out = np.empty(nbytes, dtype=np.uint8)
    cpu_lib().synth_fill_fp4(out.ctypes.data, nbytes, seed, tid, lbase)
    return out


def cpu_e8m0_bytes(n: int, seed: int, tid: int, lbase: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.uint8)
    cpu_lib().synth_fill_e8m0(out.ctypes.data, n, seed, tid, lbase)
    return out


def mxfp4_cpu(shape: Shape, seed: int, layer: int, kind: int):
    """Stored bytes of one MXFP4 projection: codes uint8 [rows][cols/2] and block scale
    bytes uint8 [rows][cols/32] (row-major, as the library takes them unpacked)."""
    rows, cols = shape.weight_shape(kind)
    codes = cpu_fp4_bytes(rows * cols // 2, seed, fp4_code_tid(layer, kind))
    scales = cpu_e8m0_bytes(rows * cols // 32, seed, fp4_scale_tid(layer, kind))
    return codes.reshape(rows, cols // 2), scales.reshape(rows, cols // 32)


def fast_set(vocab: int, size: int, seed: int, stream: int = 7) -> np.ndarray:
    """`size` distinct token ids drawn uniformly (first distinct draws of a token stream)."""
    ids: List[int] = []
    seen = set()
    base = 0
    while len(ids) < size:
        for t in cpu_tokens(4 * size, seed, stream, vocab, lbase=base).tolist():
            if t not in seen:
                seen.add(t)
                ids.append(t)
                if len(ids) == size:
                    break
        base += 4 * size
    return np.array(ids, dtype=np.int32)


def bitmap_from_ids(vocab: int, ids: Sequence[int]) -> np.ndarray:
    """Fast-answer set as a bitmap: bit (t & 31) of word (t >> 5)."""
    words = np.zeros((vocab + 31) // 32, dtype=np.uint32)
    for t in ids:
        words[int(t) >> 5] |= np.uint32(1) << np.uint32(int(t) & 31)
    return words


def weight_cpu(shape: Shape, seed: int, layer: int, kind: int) -> np.ndarray:
    """One layer weight as float32, values exactly those stored on the device (norm
    gains, and projections of models stored in their dtype; see mxfp4_cpu otherwise)."""
    if shape.mxfp4 and kind not in (ATTN_NORM, MLP_NORM):
        raise ValueError("the projections of an MXFP4 model are stored as codes: mxfp4_cpu")
    n = shape.weight_numel()[kind]
    if kind in (ATTN_NORM, MLP_NORM):
        v = cpu_values(n, seed, layer_tid(layer, kind), NORM_SIGMA, 1.0, shape.bf16)
    else:
        v = cpu_values(n, seed, layer_tid(layer, kind), WEIGHT_SIGMA, 0.0, shape.bf16)
    return v.reshape(shape.weight_shape(kind))


def global_cpu(shape: Shape, seed: int, which: int) -> np.ndarray:
    d, V = shape.d_model, shape.vocab
    if which == EMBED:
        return cpu_values(V * d, seed, EMBED, WEIGHT_SIGMA, 0.0, shape.bf16).reshape(V, d)
    if which == FINAL_NORM:
        return cpu_values(d, seed, FINAL_NORM, NORM_SIGMA, 1.0, shape.bf16)
    if which == LM_HEAD:
        return cpu_values(V * d, seed, LM_HEAD, WEIGHT_SIGMA, 0.0, shape.bf16).reshape(V, d)
    raise ValueError(which)


def lm_bias(shape: Shape, beta: float, token: int) -> np.ndarray:
    b = np.zeros(shape.vocab, dtype=np.float32)
    if beta:
        b[token] = np.float32(beta)
    return b


def kv_cpu(shape: Shape, seed: int, session: int, layer: int, which: int, head: int,
           n: int) -> np.ndarray:
    """Synthetic KV cells [n, head_dim] (float32 of the stored values) of one kv head."""
    dh = shape.head_dim
    base = (head << POS_BITS) * dh
    return cpu_values(n * dh, seed, kv_tid(session, layer, which), KV_SIGMA, 0.0, shape.bf16,
                      lbase=base).reshape(n, dh)


# ----------------------------------------------------------------------------------------
# GPU generator


def gpu_lib():
    global _gpu
    if _gpu is None:
        if not os.path.exists(GPU_LIB):
            raise RuntimeError(f"{GPU_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(GPU_LIB)
        lib.synth_gpu_fill.argtypes = [ctypes.c_void_p, ctypes.c_int] + [ctypes.c_int64] * 10 + \
            [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double, ctypes.c_float, ctypes.c_void_p]
        lib.synth_gpu_fill.restype = ctypes.c_int
        lib.synth_gpu_fill_bytes.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                             ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                                             ctypes.c_void_p]
        lib.synth_gpu_fill_bytes.restype = ctypes.c_int
        _gpu = lib
    return _gpu


def gpu_fill(ptr: int, bf16: bool, dims, lstrides, lbase: int, pstrides, seed: int, tid: int,
             sigma: float, offset: float = 0.0, stream: Optional[int] = None) -> None:
    """Generate a logical box straight into device memory at `ptr` (see synth_gpu.hip)."""
    d = list(dims) + [1] * (3 - len(dims))
    ls = list(lstrides) + [0] * (3 - len(lstrides))
    ps = list(pstrides) + [0] * (3 - len(pstrides))
    rc = gpu_lib().synth_gpu_fill(ctypes.c_void_p(ptr), 1 if bf16 else 0, d[0], d[1], d[2],
                                  ls[0], ls[1], ls[2], lbase, ps[0], ps[1], ps[2], seed, tid,
                                  sigma, offset, ctypes.c_void_p(stream or 0))
    if rc != 0:
        raise RuntimeError(f"synth_gpu_fill failed with hipError {rc}")


def gpu_fill_bytes(ptr: int, kind: int, n: int, seed: int, tid: int, lbase: int = 0,
                   stream: Optional[int] = None) -> None:
    """kind 0: n 4-bit code bytes (as cpu_fp4_bytes); kind 1: n scale bytes (as
    cpu_e8m0_bytes), straight into device memory at `ptr`."""
    rc = gpu_lib().synth_gpu_fill_bytes(ctypes.c_void_p(ptr), kind, n, lbase, seed, tid,
                                        ctypes.c_void_p(stream or 0))
    if rc != 0:
        raise RuntimeError(f"synth_gpu_fill_bytes failed with hipError {rc}")


def gpu_fill_contiguous(ptr: int, n: int, bf16: bool, seed: int, tid: int, sigma: float,
                        offset: float = 0.0, lbase: int = 0, stream: Optional[int] = None) -> None:
    gpu_fill(ptr, bf16, (n,), (1,), lbase, (1,), seed, tid, sigma, offset, stream)


# ----------------------------------------------------------------------------------------
# synthetic models and KV cells on the GPU (torch tensors filled by the GPU generator)

_KIND_NAMES = {ATTN_NORM: "attn_norm", WQ: "wq", WK: "wk", WV: "wv", WO: "wo",
               MLP_NORM: "mlp_norm", WG: "w_gate", WU: "w_up", WD: "w_down"}


def gpu_weights(shape: Shape, seed: int, lm_bias_vec: Optional[np.ndarray] = None,
                device: str = "cuda") -> dict:
    """Every weight of `shape` as a device tensor (bf16 or fp32), values identical to
    ``weight_cpu`` / ``global_cpu``.  Per-layer weights are lists under the spp key names."""
    import torch
    dt = torch.bfloat16 if shape.bf16 else torch.float32

    def make(n: int, tid: int, sigma: float, offset: float):
        t = torch.empty(n, dtype=dt, device=device)
        gpu_fill_contiguous(t.data_ptr(), n, shape.bf16, seed, tid, sigma, offset)
        return t

    d, V = shape.d_model, shape.vocab
    w = {"embed": make(V * d, EMBED, WEIGHT_SIGMA, 0.0),
         "final_norm": make(d, FINAL_NORM, NORM_SIGMA, 1.0),
         "lm_head": make(V * d, LM_HEAD, WEIGHT_SIGMA, 0.0)}
    if lm_bias_vec is not None:
        w["lm_bias"] = torch.from_numpy(np.ascontiguousarray(lm_bias_vec, dtype=np.float32)).to(device)
    numel = shape.weight_numel()

    def make_bytes(n: int, kind: int, tid: int):
        t = torch.empty(n, dtype=torch.uint8, device=device)
        gpu_fill_bytes(t.data_ptr(), kind, n, seed, tid)
        return t

    if shape.mxfp4:
        w["scales"] = {}
    for kind, name in _KIND_NAMES.items():
        norm = kind in (ATTN_NORM, MLP_NORM)
        if shape.mxfp4 and not norm:
            w[name] = [make_bytes(numel[kind] // 2, 0, fp4_code_tid(l, kind))
                       for l in range(shape.n_layers)]
            w["scales"][name] = [make_bytes(numel[kind] // 32, 1, fp4_scale_tid(l, kind))
                                 for l in range(shape.n_layers)]
            continue
        w[name] = [make(numel[kind], layer_tid(l, kind), NORM_SIGMA if norm else WEIGHT_SIGMA,
                        1.0 if norm else 0.0) for l in range(shape.n_layers)]
    torch.cuda.synchronize()
    return w


def gpu_fill_kv(base_ptr: int, layout, shape: Shape, seed: int, session: int, layer: int,
                n: int, stream: Optional[int] = None) -> None:
    """Synthetic cells [0, n) of one layer, written through a (head, position, dim) layout
    {k_offset, v_offset, k_stride[3], v_stride[3], elem_bytes}: values equal ``kv_cpu``."""
    dh = shape.head_dim
    lstr = ((1 << POS_BITS) * dh, dh, 1)
    for which, off, strides in ((0, layout.k_offset, layout.k_stride),
                                (1, layout.v_offset, layout.v_stride)):
        gpu_fill(base_ptr + off, shape.bf16, (shape.n_kv, n, dh), lstr, 0,
                 tuple(strides[i] for i in range(3)), seed, kv_tid(session, layer, which),
                 KV_SIGMA, 0.0, stream)


# ----------------------------------------------------------------------------------------
# workload recipes: the entry of decision point k, the persistent cells, the planted bias

PREFILL_STREAM, PREFIX_STREAM, HEADER_STREAM, ENVELOPE_STREAM, TARGET_STREAM, TINY_STREAM = \
    0, 1, 2, 3, 4, 5
HEADER_LEN = 8


def batched_spec(n_sessions: int, seed: int, n_range=(1024, 8192), m_range=(8, 64)):
    """(resident cells, entry length) per session of the batched workload: uniform integer
    draws n in [n_range], M in [m_range] from two token streams of `seed`."""
    n = cpu_tokens(n_sessions, seed, 900, n_range[1] - n_range[0] + 1) + n_range[0]
    m = cpu_tokens(n_sessions, seed, 901, m_range[1] - m_range[0] + 1) + m_range[0]
    return [(int(a), int(b)) for a, b in zip(n, m)]


def batched_entry(seed: int, session: int, length: int, vocab: int) -> np.ndarray:
    """Entry tokens of session `session` of the batched workload (uniform ids)."""
    return cpu_tokens(length, seed, 1000 + session, vocab)


def entry_tokens(wl: Workload, k: int = 0) -> np.ndarray:
    """Entry of decision point k: streaming = query prefix (k-th draw) + a fixed assistant
    header of 8 ids; agentic = a post-tool-call envelope; others = uniform ids."""
    V = wl.shape.vocab
    if wl.name in ("stream8b", "stream70b_mxfp4"):
        prefix = cpu_tokens(wl.entry_len - HEADER_LEN, wl.seed, PREFIX_STREAM, V,
                            lbase=k * (wl.entry_len - HEADER_LEN))
        return np.concatenate([prefix, cpu_tokens(HEADER_LEN, wl.seed, HEADER_STREAM, V)])
    stream = {"agentic8b": ENVELOPE_STREAM, "target32b": TARGET_STREAM}.get(wl.name, TINY_STREAM)
    return cpu_tokens(wl.entry_len, wl.seed, stream, V, lbase=k * wl.entry_len)


def prefill_tokens(wl: Workload) -> np.ndarray:
    """The real prefill that builds the persistent cells of a workload without synthetic KV."""
    return cpu_tokens(wl.n_past, wl.seed, PREFILL_STREAM, wl.shape.vocab)


def planted_token(wl: Workload) -> int:
    """Token that carries the logit bias beta (the first fast-answer id)."""
    return int(fast_set(wl.shape.vocab, wl.fast_set_size, wl.seed)[0])


def workload_bias(wl: Workload, beta: Optional[float] = None) -> Optional[np.ndarray]:
    beta = wl.lm_bias if beta is None else beta
    if not beta:
        return None
    return lm_bias(wl.shape, beta, planted_token(wl))
