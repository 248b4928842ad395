"""The per-kernel profile of a pre-position (spp_profile_preposition): a real pass with the
plain pass's effects, and one timed entry per kernel launch, each in its kernel's class."""
import pytest

import synth
from gpu_util import build_model, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_profiled_pass_equals_the_plain_pass_and_times_every_kernel(dtype):
    import torch
    import paper_2606_29565_amd as spp
    shape = synth.TINY.with_dtype(dtype) if dtype == "bf16" else synth.TINY
    b = build_model(shape, 41, max_tokens=64)
    toks = synth.cpu_tokens(40, 41, 0, shape.vocab).tolist()
    plain, profiled = spp.Session(b.model, 64), spp.Session(b.model, 64)
    for s in (plain, profiled):
        s.append_delta(toks[:24])
    d0 = torch.empty(shape.vocab, dtype=torch.float32, device="cuda")
    d1 = torch.empty_like(d0)
    plain.preposition(toks[24:], d0)
    prof = b.model.profile_preposition(profiled, toks[24:], d1)
    torch.cuda.synchronize()
    assert torch.equal(d0, d1)
    L = shape.n_layers
    counts = {k: v[1] for k, v in prof.items()}
    log(f"{dtype} profile: " + ", ".join(f"{k} {v[0]:.1f} us/{v[1]}" for k, v in prof.items()))
    # per layer: QKV projection, its epilogue, attention, key-range merge, O projection,
    # two residual reductions, gate/up projection, down projection; once: the LM head and
    # the merge of its partials.  40 cells are one 64-key block per kv head: a bf16 model's
    # single work item writes the attention output itself and no merge is launched
    merges = L if dtype == "f32" else 0
    for k, n in {"gemm_qkv": L, "qkv_epilogue": L, "attention": L, "attention_combine": merges,
                 "gemm_o": L, "residual_norm": 2 * L, "gemm_gate_up": L, "gemm_down": L,
                 "lm_head": 2}.items():
        assert counts[k] == n, (k, counts[k], n)
    assert counts["embed_norm"] >= 1
    assert counts["swiglu"] in (0, L) and counts["scan"] == 0
    for k, (us, n) in prof.items():
        assert (us > 0) == (n > 0), (k, us, n)
    # the profiling pass left the session as a plain pass does: a next pass agrees too
    plain.preposition(toks[24:36], d0)
    profiled.preposition(toks[24:36], d1)
    torch.cuda.synchronize()
    assert torch.equal(d0, d1)
    # an entry beyond the headroom (a skip for spp_preposition) is an error here
    with pytest.raises(spp.SppError, match="headroom"):
        b.model.profile_preposition(profiled, (toks + toks)[:41], d1)
    plain.close()
    profiled.close()
