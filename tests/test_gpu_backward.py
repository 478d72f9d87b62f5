"""GPU parity of the backward pass (tm_sparse_causal_attn_bwd) against the
oracle (``oracle.full_sequence_attention_backward``, fp64 on the same bf16
values).

The device path is the training step: the full-sequence forward (giving o and
the log-sum-exp) followed by the backward on the same inputs; the oracle
computes the gradients from q, k, v and dO alone. dq, dk and dv are each
compared element by element with
    |err| <= 2e-2 x RMS(compared tensor) + 2^-8 |g| + 2^-8 m,
where g is the oracle's gradient and m the oracle's sum of absolute products
behind it (scale |dS||K|, scale |dS|^T|Q|, |P|^T|dO|). The second term is the
bf16 rounding of the result. The third bounds the rounding of P and dS to bf16
for the MFMAs (relative error 2^-9 per factor, doubled): dS sums to zero over
a row, so a gradient is a sum of products of both signs and its rounding
error scales with m, not with |g|. CPU emulation of this arithmetic stays
within 0.45 of the bound; a missing delta term, a missing scale, an
untransposed P or a 5% error in P exceed it 4-950 times. Geometries: ragged query and key tiles, W = 0, 1, 2, a
three-frame c_0, D = 64 and 128, batch 2, and a 21-frame sequence with the
480p chunk structure (R = 1, C = 3) at 256 tokens per frame.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import say
from oracle import ChunkGeometry, full_sequence_attention_backward
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
    return bf16_bits_to_f32(bits), torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def _run(tm, seed, B, H, D, T, C, R, W, frames, heads=None):
    rng = np.random.default_rng(seed)
    L = frames * T
    (q, qd), (k, kd), (v, vd) = (_bf16(rng, (B, L, H, D), i < 2) for i in range(3))
    do, dod = _bf16(rng, (B, L, H, D), False)
    desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
    lse = torch.empty(B, H, L, dtype=torch.float32, device="cuda")
    o = tm.tm_sparse_causal_attn_fwd(desc, qd, -1, k=kd, v=vd, n_frames=frames, lse=lse)
    dq, dk, dv = tm.tm_sparse_causal_attn_bwd(desc, frames, qd, kd, vd, o, lse, dod)
    torch.cuda.synchronize()
    g = ChunkGeometry(T, C, R, W)
    want, mags = full_sequence_attention_backward(q, k, v, do, g, heads=heads, magnitudes=True)
    got = [x.float().cpu().numpy() for x in (dq, dk, dv)]
    if heads is not None:
        got = [x[:, :, heads] for x in got]
    return got, want, mags


def _assert_grad(got, want, mag, what):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite gradient"
    rms = float(np.sqrt(np.mean(want ** 2)))
    bound = 2e-2 * rms + 2.0 ** -8 * np.abs(want) + 2.0 ** -8 * mag
    worst = float(np.max(np.abs(got - want) / bound))
    say(f"  {what}: max|err| / rms = {np.max(np.abs(got - want)) / rms:.2e}, worst err / bound = {worst:.3f}")
    assert worst <= 1.0, f"{what}: error {worst:.3f} x the bound"


@pytest.mark.parametrize("T,C,R,W,frames,D", [
    (16, 2, 1, 1, 9, 128),    # 144 tokens: one query tile per chunk, keys in one tile
    (50, 3, 1, 1, 7, 64),     # ragged tiles, D = 64
    (40, 2, 3, 2, 11, 128),   # three-frame c_0, W = 2
    (20, 3, 1, 0, 7, 128),    # W = 0: each chunk sees c_0 and itself
    (130, 3, 1, 1, 7, 128),   # chunks of 390 rows: 4 query tiles (last 6 rows), 2 key tiles
    (40, 2, 3, 1, 3, 128),    # the reference chunk alone: only c_0 tiles in both grids
    (16, 2, 1, 1, 2, 128),    # c_0 and one frame of a two-frame chunk
])
def test_backward_matches_oracle(tm, T, C, R, W, frames, D):
    say(f"backward vs oracle: T={T} C={C} R={R} W={W} frames={frames} D={D}")
    got, want, mags = _run(tm, 7 * T + W, 2, 2, D, T, C, R, W, frames)
    for name, g_, w_, m_ in zip(("dq", "dk", "dv"), got, want, mags):
        _assert_grad(g_, w_, m_, f"{name} T={T} W={W} D={D}")


def test_backward_many_heads(tm):
    # 2 x 7 = 14 (batch, head) pairs: the grids' per-XCD grouping spans several heads
    say("backward: B=2 H=7, T=48 C=2 R=1 W=1, 7 frames")
    got, want, mags = _run(tm, 5, 2, 7, 64, 48, 2, 1, 1, 7)
    for name, g_, w_, m_ in zip(("dq", "dk", "dv"), got, want, mags):
        _assert_grad(g_, w_, m_, f"{name} B=2 H=7")


def test_backward_21_frame_sequence(tm):
    # the 480p chunk structure (c_0 = 1 frame, chunks of 3, last chunk of 2)
    # at 256 tokens per frame: 5376 tokens, 8 chunks
    say("backward: 21 frames x 256 tokens, R=1 C=3 W=1")
    got, want, mags = _run(tm, 21, 1, 2, 128, 256, 3, 1, 1, 21)
    for name, g_, w_, m_ in zip(("dq", "dk", "dv"), got, want, mags):
        _assert_grad(g_, w_, m_, f"{name} 21x256")


def test_backward_is_deterministic_and_checks_arguments(tm):
    B, H, D, T, C, R, W, frames = 1, 2, 128, 64, 2, 1, 1, 5
    rng = np.random.default_rng(5)
    L = frames * T
    _, q = _bf16(rng, (B, L, H, D), True)
    _, k = _bf16(rng, (B, L, H, D), True)
    _, v = _bf16(rng, (B, L, H, D), False)
    _, do = _bf16(rng, (B, L, H, D), False)
    desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
    lse = torch.empty(B, H, L, dtype=torch.float32, device="cuda")
    o = tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=frames, lse=lse)
    g1 = tm.tm_sparse_causal_attn_bwd(desc, frames, q, k, v, o, lse, do)
    g2 = tm.tm_sparse_causal_attn_bwd(desc, frames, q, k, v, o, lse, do)
    torch.cuda.synchronize()
    for a, b in zip(g1, g2):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    with pytest.raises(tm.TMError) as e:  # dq may not be q
        tm.tm_sparse_causal_attn_bwd(desc, frames, q, k, v, o, lse, do, dq=q)
    assert e.value.status == tm.TM_E_ARG
    with pytest.raises(tm.TMError) as e:  # too few rows for the frames asked
        tm.tm_sparse_causal_attn_bwd(desc, frames + 1, q, k, v, o, lse, do)
    assert e.value.status == tm.TM_E_ARG


def _chunk_tile_rows(g, L, tile, per_chunk, rng):
    """In every chunk: its first two and last two rows, both rows at each of
    its first three and last three tile boundaries (tiles are chunk-aligned, so
    the last tile of a chunk is its ragged tail), and ``per_chunk`` random rows."""
    from oracle.attention import chunk_start
    rows = set()
    a = 0
    while chunk_start(a, g) < L:
        lo, hi = chunk_start(a, g), min(chunk_start(a + 1, g), L)
        rows.update({lo, lo + 1, hi - 2, hi - 1})
        bounds = list(range(lo + tile, hi, tile))
        for b in bounds[:3] + bounds[-3:]:
            rows.update({b - 1, b})
        rows.update(rng.choice(np.arange(lo, hi), size=per_chunk, replace=False).tolist())
        a += 1
    return np.array(sorted(rows))


def test_backward_480p_full_sequence_sampled(tm):
    """The shape the benchmark times: 21 latent frames x 1560 tokens (c_0 of one
    frame, six chunks of 3 frames, one of 2), D = 128, two heads. Query tiles
    of 128 rows leave tails of 24 (c_0), 72 (3-frame chunks) and 48 rows (the
    last chunk); key tiles likewise. The oracle computes dQ for rows sampled in
    every chunk and dK/dV for keys sampled in every chunk, each over complete
    masked rows (``sampled_sequence_attention_backward``), head 1 of 2."""
    from oracle.backward import sampled_sequence_attention_backward
    from synth import draw_qkv_sequence, draw_tensor
    from synth.inputs import FULL_SEQUENCE_CHUNK, Workload

    B, H, D, T, C, R, W, frames = 1, 2, 128, 1560, 3, 1, 1, 21
    L = frames * T
    w = Workload(460, "bwd_480p", "bf16", B, H, D, T, C, R, W, n_frames=frames)
    d = draw_qkv_sequence(w)
    do, do_bits = draw_tensor((L, H, D), wid=w.wid, b=0, chunk=FULL_SEQUENCE_CHUNK, step=0,
                              layer=0, tensor_id=3, rms_normalise=False, dtype="bf16")
    dev = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(
        torch.bfloat16).cuda()
    qd, kd, vd = (dev(d[n + "_bits"]) for n in "qkv")
    dod = dev(do_bits[None])
    desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
    say("backward 480p: forward + backward, 21 x 1560 tokens, 2 heads")
    lse = torch.empty(B, H, L, dtype=torch.float32, device="cuda")
    o = tm.tm_sparse_causal_attn_fwd(desc, qd, -1, k=kd, v=vd, n_frames=frames, lse=lse)
    dq, dk, dv = tm.tm_sparse_causal_attn_bwd(desc, frames, qd, kd, vd, o, lse, dod)
    torch.cuda.synchronize()
    g = ChunkGeometry(T, C, R, W)
    rng = np.random.default_rng(21)
    q_rows = _chunk_tile_rows(g, L, 128, 6, rng)
    k_rows = _chunk_tile_rows(g, L, 128, 6, rng)
    say(f"backward 480p oracle: {len(q_rows)} dQ rows, {len(k_rows)} dK/dV rows, head 1")
    (wq, wk, wv), (mq, mk, mv) = sampled_sequence_attention_backward(
        d["q"], d["k"], d["v"], do[None], g, q_rows=q_rows, k_rows=k_rows, heads=[1])
    got_q = dq.float().cpu().numpy()[:, q_rows][:, :, [1]]
    got_k = dk.float().cpu().numpy()[:, k_rows][:, :, [1]]
    got_v = dv.float().cpu().numpy()[:, k_rows][:, :, [1]]
    _assert_grad(got_q, wq, mq, "dq 480p")
    _assert_grad(got_k, wk, mk, "dk 480p")
    _assert_grad(got_v, wv, mv, "dv 480p")
