"""The allocation-free backward (tm_sparse_causal_attn_bwd_noalloc), whose
delta workspace is the library's device-global array, against the backward
with a caller-owned workspace (tm_sparse_causal_attn_bwd): the same kernels,
so the gradients must agree bit for bit. Two calls in a row, the second on a
smaller problem, so that the second runs over what the first left in the
array; sizes beyond the array are rejected before anything is launched.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import say
from synth import bf16_bits_to_f32, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tm():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2506_03099_amd import tm as binding
    binding.lib()
    return binding


def _bf16(rng, shape, norm):
    x = rng.standard_normal(shape).astype(np.float32)
    if norm:
        x /= np.sqrt(np.mean(x * x, axis=-1, keepdims=True))
    bits = f32_to_bf16_bits(x)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def test_noalloc_backward_equals_the_workspace_backward(tm):
    for call, (B, H, D, T, C, R, W, frames) in enumerate([(2, 3, 128, 40, 2, 1, 1, 9),
                                                          (1, 2, 64, 24, 3, 1, 1, 5)]):
        say(f"noalloc backward call {call}: B={B} H={H} D={D} T={T} frames={frames}")
        rng = np.random.default_rng(70 + call)
        L = frames * T
        q, k = _bf16(rng, (B, L, H, D), True), _bf16(rng, (B, L, H, D), True)
        v, do = _bf16(rng, (B, L, H, D), False), _bf16(rng, (B, L, H, D), False)
        desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
        lse = torch.empty(B, H, L, dtype=torch.float32, device="cuda")
        o = tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=frames, lse=lse)
        want = tm.tm_sparse_causal_attn_bwd(desc, frames, q, k, v, o, lse, do)
        got = tuple(torch.full_like(q, float("nan")) for _ in range(3))
        tm.tm_sparse_causal_attn_bwd_noalloc(desc, frames, q, k, v, o, lse, do, *got)
        torch.cuda.synchronize()
        for name, g, w in zip(("dq", "dk", "dv"), got, want):
            same = torch.equal(g.view(torch.int16), w.view(torch.int16))
            say(f"  {name}: bitwise equal to the workspace call: {same}")
            assert same, f"call {call}: {name} differs"


def test_noalloc_rejects_problems_beyond_its_workspace(tm):
    # 64 heads x 33 frames x 1024 tokens = 2,162,688 rows > 2^21
    desc = tm.make_desc(1, 64, 64, 1024, 3, 1, 1, "bf16")
    x = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros(16, dtype=torch.float32, device="cuda")
    with pytest.raises(tm.TMError) as e:
        tm.tm_sparse_causal_attn_bwd_noalloc(desc, 33, x, x, x, x, lse, x, x, x, x)
    assert e.value.status == tm.TM_E_CAPACITY
    assert "workspace" in str(e.value)
    # exactly at the limit the size check passes (and the pointer checks then fail)
    with pytest.raises(tm.TMError) as e:
        tm.tm_sparse_causal_attn_bwd_noalloc(tm.make_desc(1, 64, 64, 1024, 3, 1, 1, "bf16"), 32,
                                             x, x, x, x, lse, x, x, x, x)
    assert e.value.status == tm.TM_E_ARG
