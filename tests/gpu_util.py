"""Helpers for the GPU tests: synthetic models on the device, KV readback, oracle runs."""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

import oracle
import synth


def log(*a):
    print(*a, flush=True)


@dataclasses.dataclass
class Built:
    shape: synth.Shape
    seed: int
    model: object
    weights: dict
    bias: Optional[np.ndarray]


def build_model(shape: synth.Shape, seed: int, bias: Optional[np.ndarray] = None,
                max_tokens: int = 128, max_sessions: int = 1, packed: bool = False) -> Built:
    """A synthetic model on cuda:0 behind the C ABI.  packed=True hands the library
    tiled projection weights made with spp_pack_weight (else it packs its own copies)."""
    import torch
    import paper_2606_29565_amd as spp
    w = synth.gpu_weights(shape, seed, bias)
    if packed:
        cfg = spp.model_config(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim,
                               shape.ffn, shape.vocab, shape.rope_base, shape.bf16,
                               rms_eps=shape.eps, max_tokens=max_tokens,
                               max_sessions=max_sessions, weights_packed=True,
                               mxfp4=shape.mxfp4)
        kinds = {"wq": spp.SPP_W_Q, "wk": spp.SPP_W_K, "wv": spp.SPP_W_V, "wo": spp.SPP_W_O,
                 "w_gate": spp.SPP_W_GATE, "w_up": spp.SPP_W_UP, "w_down": spp.SPP_W_DOWN}
        for key, which in kinds.items():
            tiled, tiled_sc = [], []
            for i, t in enumerate(w[key]):
                dst = torch.empty_like(t)
                if shape.mxfp4:
                    sc = w["scales"][key][i]
                    dst_sc = torch.empty_like(sc)
                    spp.pack_weight_mxfp4(cfg, which, t, sc, dst, dst_sc)
                    tiled_sc.append(dst_sc)
                else:
                    spp.pack_weight(cfg, which, t, dst)
                tiled.append(dst)
            w[key] = tiled
            if shape.mxfp4:
                w["scales"][key] = tiled_sc
        torch.cuda.synchronize()
    m = spp.Model(shape.n_layers, shape.d_model, shape.n_q, shape.n_kv, shape.head_dim, shape.ffn,
                  shape.vocab, shape.rope_base, shape.bf16, w, rms_eps=shape.eps,
                  max_tokens=max_tokens, max_sessions=max_sessions, weights_packed=packed,
                  mxfp4=shape.mxfp4)
    return Built(shape, seed, m, w, bias)


def fill_synthetic_kv(b: Built, sess, session_id: int, n: int) -> None:
    for l in range(b.shape.n_layers):
        synth.gpu_fill_kv(sess.kv.data_ptr(), b.model.kv_layout(sess.capacity, l), b.shape, b.seed,
                          session_id, l, n)


def read_kv(b: Built, sess, layer: int, n: int):
    """Cells [0, n) of one layer as float32 arrays K, V of shape [n_kv, n, head_dim]."""
    import torch
    s = b.shape
    lay = b.model.kv_layout(sess.capacity, layer)
    eb = lay.elem_bytes
    dt = torch.bfloat16 if s.bf16 else torch.float32
    kv = sess.kv
    k = kv[lay.k_offset: lay.k_offset + s.n_kv * lay.k_stride[0] * eb].view(dt)
    k = k.view(s.n_kv, -1, s.head_dim)[:, :n].float().cpu().numpy()
    v = kv[lay.v_offset: lay.v_offset + s.n_kv * lay.v_stride[0] * eb].view(dt)
    v = v.view(s.n_kv, s.head_dim, -1)[:, :, :n].float().cpu().numpy().transpose(0, 2, 1)
    return k, v


def oracle_logits(shape: synth.Shape, seed: int, n_past: int, entry: Sequence[int],
                  prefill: Optional[Sequence[int]] = None, kv_synth: bool = False,
                  session: int = 0, bias: Optional[np.ndarray] = None, last_only: bool = False,
                  kv_out: Optional[list] = None) -> np.ndarray:
    """The oracle's ready distribution for `entry` at n_past; the persistent cells are
    either a real prefill of `prefill` (n_past tokens) or synthetic draws."""
    w = oracle.Weights(shape, seed, lm_bias=bias, cache_layers=shape.n_layers <= 4)
    cap = n_past + len(entry)
    kv = oracle.KVState(shape, cap, seed=seed, session=session,
                        n_synth=n_past if kv_synth else 0)
    if prefill is not None and n_past:
        oracle.forward(w, kv, 0, prefill, logits=False)
    out = oracle.forward(w, kv, n_past, entry, last_only=last_only)
    if kv_out is not None:
        kv_out.append(kv)
    return out


def max_abs(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
