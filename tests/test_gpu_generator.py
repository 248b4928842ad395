"""The GPU implementation of the seeded generator equals the CPU one bit for bit, for
contiguous tensors and for a strided KV layout (so both sides of every parity test see
identical inputs)."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("bf16", [False, True])
def test_gpu_fill_matches_cpu(bf16):
    import torch
    n = 300_001
    for tid, sigma, offset, lbase in ((5, 0.02, 0.0, 0), (9, 1.0, 0.0, 12345), (7, 0.02, 1.0, 3)):
        t = torch.empty(n, dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
        synth.gpu_fill_contiguous(t.data_ptr(), n, bf16, 42, tid, sigma, offset, lbase=lbase)
        got = t.float().cpu().numpy()
        ref = synth.cpu_values(n, 42, tid, sigma, offset, bf16, lbase=lbase)
        np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_gpu_fill_strided_kv_box():
    import torch
    shape = synth.Shape("kvbox", 1, 64, 4, 2, 64, 128, 256, 1e4, "bf16")
    n, cap = 37, 64
    buf = torch.zeros(2 * shape.n_kv * cap * shape.head_dim, dtype=torch.bfloat16, device="cuda")

    class L:  # K as [head][pos][dim], V transposed as [head][dim][pos]
        k_offset = 0
        v_offset = shape.n_kv * cap * shape.head_dim * 2
        k_stride = (cap * shape.head_dim, shape.head_dim, 1)
        v_stride = (shape.head_dim * cap, 1, cap)
        elem_bytes = 2

    synth.gpu_fill_kv(buf.data_ptr(), L, shape, 42, 3, 0, n)
    torch.cuda.synchronize()
    half = shape.n_kv * cap * shape.head_dim
    K = buf[:half].view(shape.n_kv, cap, shape.head_dim)[:, :n].float().cpu().numpy()
    V = buf[half:].view(shape.n_kv, shape.head_dim, cap)[:, :, :n].float().cpu().numpy()
    for h in range(shape.n_kv):
        np.testing.assert_array_equal(K[h], synth.kv_cpu(shape, 42, 3, 0, 0, h, n))
        np.testing.assert_array_equal(V[h].T, synth.kv_cpu(shape, 42, 3, 0, 1, h, n))
    assert float(buf[:half].view(shape.n_kv, cap, -1)[:, n:].abs().max()) == 0.0
