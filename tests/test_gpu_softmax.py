"""GPU parity of the online softmax where its running maximum must rise.

With unit-RMS queries and keys and the scale 1/sqrt(D), a logit in the log2
domain is at most 1.44 sqrt(D) (16.3 at D = 128), so the bf16 kernel's lazy
maximum (taken exactly on the first key tile, raised only when a later score
exceeds it by more than 16 in the log2 domain) never has to rise. Here the
inputs are built so that it must (``synth.draw_rising_sequence``): the keys
after c_0 score 2 u + r against queries 2 u + r' with a weight that grows
along the sequence, so every query row past c_0 sees scores 30-90 above its
first tile's maximum. The test asserts that property on the CPU before the
comparison, so the rescale of O and of the row sums, the shift of the scores
and the re-formed P all run, several times per row, in the cache form (V^T
from dimension-major blocks) and the whole-sequence form (row-major V), at
D = 64 and 128, and in the fp32 kernel. A second group passes a softmax scale
of 8 / sqrt(D) through the descriptor on random inputs.

Bar: the bf16 kernel's arithmetic, through its fp32 output, within 2e-2 x RMS
of the oracle, and its bf16 output equal to that fp32 output rounded to
nearest even, bit for bit; fp32 within 1e-4 x RMS; the log-sum-exp within
``LSE_ATOL`` (1e-4) of the oracle's: the row sums are formed in fp32 from the
unrounded P.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import LSE_ATOL, assert_close, assert_rounds_to, from_dev, say, to_dev
from oracle import ChunkGeometry, StreamHistory, full_sequence_attention
from oracle.attention import chunk_start
from synth import draw_qkv_sequence
from synth.inputs import Workload, draw_rising_sequence

pytestmark = pytest.mark.gpu

LOG2E = float(np.log2(np.e))


@pytest.fixture(scope="module")
def tm():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2506_03099_amd import tm as binding
    binding.lib()
    return binding


def _rise_above_first_tile(q, k, g, scale, L):
    """Smallest, over query rows past c_0, of (largest allowed score - largest
    score of the first 64 keys), log2 domain; the kernels visit keys 0..63 of
    c_0 first."""
    from oracle import allowed_mask
    worst = np.inf
    pos = np.arange(L)
    rows = pos[pos >= chunk_start(1, g)]
    mask = allowed_mask(rows, pos, g)
    for b in range(q.shape[0]):
        for h in range(q.shape[2]):
            s = (q[b, rows, h].astype(np.float64) @ k[b, :, h].T.astype(np.float64)) * scale * LOG2E
            first = s[:, :64].max(axis=1)
            top = np.where(mask, s, -np.inf).max(axis=1)
            worst = min(worst, float((top - first).min()))
    return worst


def _upload(d, dtype):
    return tuple(to_dev(d[n], d.get(n + "_bits"), dtype) for n in "qkv")


RISING = [
    # name, dtype, B, H, D, T, C, R, W, frames
    ("d128", "bf16", 1, 2, 128, 64, 2, 1, 1, 9),
    ("d64_ragged", "bf16", 2, 2, 64, 50, 3, 2, 1, 10),
    ("d128_w2", "bf16", 1, 3, 128, 40, 2, 2, 2, 11),
    ("d128_f32", "f32", 1, 2, 128, 64, 2, 1, 1, 9),
    ("d64_f32", "f32", 1, 2, 64, 50, 3, 2, 1, 10),
]


def _rising(case, seed):
    name, dtype, B, H, D, T, C, R, W, frames = case
    g = ChunkGeometry(T, C, R, W)
    L = frames * T
    d = draw_rising_sequence(seed, B, L, H, D, cold_tokens=R * T, gamma_lo=2.0, gamma_hi=6.0,
                             dtype=dtype)
    rise = _rise_above_first_tile(d["q"], d["k"], g, 1 / np.sqrt(D), L)
    say(f"rising {name}: every row past c_0 scores >= {rise:.1f} (log2) above its first tile")
    assert rise > 17.0, "the construction no longer forces the running maximum up"
    return g, L, d


def _check(tm, desc, dtype, run, run_f32, want, lse, lse_ref, what):
    """run() -> bf16 (or fp32) output; run_f32() -> fp32 output of the same call."""
    o = run()
    if dtype == "bf16":
        of = run_f32()
        torch.cuda.synchronize()
        assert_rounds_to(o, of, what)
        assert_close(from_dev(of), want, "bf16", what)
    else:
        torch.cuda.synchronize()
        assert_close(from_dev(o), want, "f32", what)
    if lse is not None:
        np.testing.assert_allclose(from_dev(lse), lse_ref, rtol=0,
                                   atol=LSE_ATOL[dtype])


@pytest.mark.parametrize("case", RISING, ids=[c[0] for c in RISING])
def test_running_max_rises_whole_sequence(tm, case):
    name, dtype, B, H, D, T, C, R, W, frames = case
    g, L, d = _rising(case, 400 + len(name))
    q, k, v = _upload(d, dtype)
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype)
    lse = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    want, lse_ref = full_sequence_attention(d["q"], d["k"], d["v"], g)
    _check(tm, desc, dtype,
           lambda: tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=frames, lse=lse),
           lambda: tm.tm_sparse_causal_attn_fwd_f32out(desc, q, -1, k=k, v=v, n_frames=frames),
           want, lse, lse_ref, f"rising sequence {name}")


@pytest.mark.parametrize("case", RISING, ids=[c[0] for c in RISING])
def test_running_max_rises_from_the_cache(tm, case):
    name, dtype, B, H, D, T, C, R, W, frames = case
    g, L, d = _rising(case, 500 + len(name))
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    n_chunks = 1 + -(-(L - R * T) // (C * T))
    for t in range(n_chunks):
        lo, hi = chunk_start(t, g), min(chunk_start(t + 1, g), L)
        part = {key: val[:, lo:hi] for key, val in d.items()}
        q, k, v = _upload(part, dtype)
        tm.tm_kv_append(cache, t, k, v)
        hist.append(t, part["k"], part["v"])
        lse = torch.empty((B, H, hi - lo), dtype=torch.float32, device="cuda")
        want, lse_ref = hist.attend(part["q"], t)
        _check(tm, desc, dtype,
               lambda: tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=cache, lse=lse),
               lambda: tm.tm_sparse_causal_attn_fwd_f32out(desc, q, t, cache=cache),
               want, lse, lse_ref, f"rising cache {name} chunk {t}")


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("bf16", 64), ("f32", 128)])
def test_softmax_scale_through_the_descriptor(tm, dtype, D):
    """scale = 8 / sqrt(D): logits with a standard deviation of 8 on random
    unit-RMS inputs, both forms; the oracle takes the same scale."""
    B, H, T, C, R, W, frames = 1, 2, 48, 3, 1, 1, 10
    scale = 8.0 / np.sqrt(D)
    w = Workload(450 + D, f"scale8_{dtype}_{D}", dtype, B, H, D, T, C, R, W, n_frames=frames)
    g = ChunkGeometry(T, C, R, W)
    d = draw_qkv_sequence(w)
    q, k, v = _upload(d, dtype)
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype, softmax_scale=float(np.float32(scale)))
    L = frames * T
    lse = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    want, lse_ref = full_sequence_attention(d["q"], d["k"], d["v"], g, scale=np.float32(scale))
    say(f"softmax scale {scale:.4f}: {dtype} D={D}")
    _check(tm, desc, dtype,
           lambda: tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=frames, lse=lse),
           lambda: tm.tm_sparse_causal_attn_fwd_f32out(desc, q, -1, k=k, v=v, n_frames=frames),
           want, lse, lse_ref, f"scale 8/sqrt(D) {dtype} D={D}")
    # the cache form with the same scale
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    for t in range(4):
        lo, hi = chunk_start(t, g), min(chunk_start(t + 1, g), L)
        part = {key: val[:, lo:hi] for key, val in d.items()}
        qc, kc, vc = _upload(part, dtype)
        tm.tm_kv_append(cache, t, kc, vc)
        hist.append(t, part["k"], part["v"])
        want, _ = hist.attend(part["q"], t, scale=np.float32(scale))
        _check(tm, desc, dtype,
               lambda: tm.tm_sparse_causal_attn_fwd(desc, qc, t, cache=cache),
               lambda: tm.tm_sparse_causal_attn_fwd_f32out(desc, qc, t, cache=cache),
               want, None, None, f"scale 8/sqrt(D) cache {dtype} D={D} chunk {t}")
