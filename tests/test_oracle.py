"""Pins of the CPU oracle against what the paper and the mathematics fix.

The paper prints no worked numeric example, so the oracle is pinned by:
the chunk-level pattern written by hand from Sec. 4.2 (golden files), closed
forms for the allowed-pair counts, row sums, brute force in fp64 on tiny
inputs, library special cases (PyTorch's CPU scaled_dot_product_attention for
dense, token-causal and block-causal attention; scipy's logsumexp), constant-V
and zero-Q closed forms, invariance to disallowed keys, the statistical output
RMS, and the streaming form agreeing with the full-sequence form.
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import (ChunkGeometry, StreamHistory, allowed_mask, allowed_pair_count,
                    brute_force_attention, chunk_of_frame, full_sequence_attention,
                    masked_attention)
from oracle.attention import chunk_start
from synth import WORKLOADS, draw_chunk, draw_qkv_sequence

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden_mask(name):
    rows, frames = [], None
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line.startswith("# frames_per_chunk:"):
                frames = [int(x) for x in line.split(":")[1].split()]
            elif line and not line.startswith("#"):
                rows.append([c == "1" for c in line])
    return np.array(rows), frames


def _rand(shape, seed, dtype=np.float32):
    return np.random.default_rng(seed).standard_normal(shape).astype(dtype)


# --------------------------------------------------------------------------- geometry


@pytest.mark.parametrize("fname,R", [("chunk_mask_21f_r3c3.txt", 3), ("chunk_mask_21f_r1c3.txt", 1)])
def test_chunk_level_pattern_matches_paper(fname, R):
    want, frames_per_chunk = _read_golden_mask(fname)
    g = ChunkGeometry(tokens_per_frame=2, chunk_frames=3, ref_frames=R, window=1)
    chunks = chunk_of_frame(np.arange(21), g)
    assert np.bincount(chunks).tolist() == frames_per_chunk
    pos = np.arange(21 * 2)
    m = allowed_mask(pos, pos, g)
    tok_chunk = chunks[pos // 2]
    n = want.shape[0]
    for a in range(n):
        for c in range(n):
            block = m[np.ix_(tok_chunk == a, tok_chunk == c)]
            assert block.all() == want[a, c] and block.any() == want[a, c], (a, c)


def test_pair_count_tiny_sequence_closed_form():
    # 9 frames of 64 tokens: c_0 = 64 tokens, then four chunks of 128.
    # keys seen: c_0 -> 64; c_1 -> 64 + 128; c_2..c_4 -> 64 + 128 + 128.
    closed = 64 * 64 + 128 * 192 + 3 * 128 * 320
    assert closed == 151_552
    g = ChunkGeometry(64, 2, 1, 1)
    assert allowed_pair_count(9 * 64, g) == closed
    assert (9 * 64) ** 2 == 331_776


def test_pair_count_480p_sequence_closed_form():
    # 21 frames x 1560 tokens: c_0 1560, c_1..c_6 4680 each, c_7 3120.
    # keys: c_0 1560; c_1 6240; c_2..c_6 1560 + 9360; c_7 1560 + 4680 + 3120.
    closed = 1560 * 1560 + 4680 * 6240 + 5 * 4680 * 10920 + 3120 * 9360
    assert closed == 316_368_000
    g = ChunkGeometry(1560, 3, 1, 1)
    assert allowed_pair_count(21 * 1560, g) == closed


def test_pair_count_literal_seven_chunks_closed_form():
    # R = C = 3: seven chunks of 4680; keys c_0 4680, c_1 9360, c_2..c_6 14040.
    closed = 4680 * 4680 + 4680 * 9360 + 5 * 4680 * 14040
    g = ChunkGeometry(1560, 3, 3, 1)
    assert allowed_pair_count(21 * 1560, g) == closed
    assert abs(closed / (21 * 1560) ** 2 - 0.3673) < 1e-3


def test_large_window_is_block_causal_and_zero_window_sees_own_chunk_and_ref():
    g_big = ChunkGeometry(4, 2, 1, 100)
    g_zero = ChunkGeometry(4, 2, 1, 0)
    pos = np.arange(4 * 9)
    ch = chunk_of_frame(pos // 4, g_big)
    # block causal, written with a Kronecker product of per-chunk blocks
    n_chunks = ch.max() + 1
    sizes = np.bincount(ch)
    tri = np.tril(np.ones((n_chunks, n_chunks), dtype=bool))
    blocks = np.block([[np.full((sizes[a], sizes[c]), tri[a, c]) for c in range(n_chunks)]
                       for a in range(n_chunks)])
    assert np.array_equal(allowed_mask(pos, pos, g_big), blocks)
    m0 = allowed_mask(pos, pos, g_zero)
    eye = np.block([[np.full((sizes[a], sizes[c]), a == c or c == 0) for c in range(n_chunks)]
                    for a in range(n_chunks)])
    assert np.array_equal(m0, eye)


# --------------------------------------------------------------------------- softmax


def test_rows_sum_to_one_and_lse_matches_logsumexp():
    g = ChunkGeometry(5, 2, 1, 1)
    L, D = 5 * 7, 16
    q, k, v = (_rand((L, D), s) for s in (1, 2, 3))
    pos = np.arange(L)
    mask = allowed_mask(pos, pos, g)
    scale = 1 / math.sqrt(D)
    o, lse, p = masked_attention(q, k, v, mask, scale, return_probs=True)
    assert np.all(np.abs(p.sum(axis=1) - 1) <= 1e-6)
    assert np.all(p[~mask] == 0)
    logits = (q.astype(np.float64) @ k.T.astype(np.float64)) * scale
    ref = scipy.special.logsumexp(np.where(mask, logits, -np.inf), axis=1)
    np.testing.assert_allclose(lse, ref, rtol=0, atol=2e-5)


# --------------------------------------------------------------------------- brute force


@pytest.mark.parametrize("T,C,R,W,frames", [
    (3, 2, 1, 1, 8),   # paper's window, partial last chunk (7 = 3*2 + 1)
    (2, 3, 1, 1, 10),  # chunks of 3 frames, tail of 0
    (2, 2, 2, 0, 9),   # no previous chunk
    (2, 1, 1, 2, 7),   # window of two previous chunks
    (4, 3, 3, 1, 9),   # literal reading, c_0 = 3 frames
])
def test_oracle_matches_fp64_brute_force(T, C, R, W, frames):
    L, D = T * frames, 8
    q, k, v = (_rand((L, D), 10 + s) for s in range(3))
    g = ChunkGeometry(T, C, R, W)
    pos = np.arange(L)
    mask = allowed_mask(pos, pos, g)
    scale = 1 / math.sqrt(D)
    bo, blse, key_sets = brute_force_attention(q, k, v, T=T, C=C, R=R, W=W)
    for i in range(L):
        assert np.flatnonzero(mask[i]).tolist() == key_sets[i]
    o32, lse32 = masked_attention(q, k, v, mask, scale)
    o64, lse64 = masked_attention(q, k, v, mask, scale, dtype=np.float64)
    np.testing.assert_allclose(o64, bo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse64, blse, rtol=0, atol=1e-12)
    np.testing.assert_allclose(o32, bo, rtol=0, atol=2e-6)
    np.testing.assert_allclose(lse32, blse, rtol=0, atol=2e-6)


def test_brute_force_with_offset_queries_matches_full_sequence_rows():
    g = ChunkGeometry(3, 2, 1, 1)
    L, D = 3 * 9, 8
    q, k, v = (_rand((1, L, 1, D), 20 + s) for s in range(3))
    o_full, _ = full_sequence_attention(q, k, v, g, dtype=np.float64)
    q_off = chunk_start(3, g)
    rows = np.arange(q_off, q_off + 6)
    bo, _, _ = brute_force_attention(q[0, rows, 0], k[0, :, 0], v[0, :, 0], T=3, C=2, R=1, W=1,
                                     q_positions=rows)
    np.testing.assert_allclose(o_full[0, rows, 0], bo, rtol=0, atol=1e-12)


# --------------------------------------------------------------------------- library special cases


def _sdpa(q, k, v, **kw):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), **kw)[0, 0].numpy()


def test_single_chunk_is_dense_attention():
    # every token inside c_0 (R frames cover the whole sequence)
    g = ChunkGeometry(4, 2, 6, 1)
    L, D = 24, 16
    q, k, v = (_rand((1, L, 1, D), 30 + s) for s in range(3))
    o, _ = full_sequence_attention(q, k, v, g, dtype=np.float64)
    np.testing.assert_allclose(o[0, :, 0], _sdpa(q[0, :, 0], k[0, :, 0], v[0, :, 0]),
                               rtol=0, atol=1e-12)


def test_one_token_chunks_with_unbounded_window_is_token_causal():
    g = ChunkGeometry(1, 1, 1, 10_000)
    L, D = 40, 16
    q, k, v = (_rand((1, L, 1, D), 40 + s) for s in range(3))
    o, _ = full_sequence_attention(q, k, v, g, dtype=np.float64)
    np.testing.assert_allclose(o[0, :, 0], _sdpa(q[0, :, 0], k[0, :, 0], v[0, :, 0], is_causal=True),
                               rtol=0, atol=1e-12)


def test_window_covering_all_chunks_is_block_causal():
    T, C = 3, 2
    g = ChunkGeometry(T, C, C, 50)  # c_0 as wide as the other chunks
    n_chunks, D = 5, 16
    L = n_chunks * C * T
    q, k, v = (_rand((1, L, 1, D), 50 + s) for s in range(3))
    o, _ = full_sequence_attention(q, k, v, g, dtype=np.float64)
    block_mask = np.kron(np.tril(np.ones((n_chunks, n_chunks))), np.ones((C * T, C * T))) > 0
    ref = _sdpa(q[0, :, 0], k[0, :, 0], v[0, :, 0], attn_mask=torch.from_numpy(block_mask))
    np.testing.assert_allclose(o[0, :, 0], ref, rtol=0, atol=1e-12)


# --------------------------------------------------------------------------- closed forms


def test_constant_v_rows_give_that_constant():
    g = ChunkGeometry(4, 2, 1, 1)
    L, D = 4 * 9, 8
    q, k = _rand((1, L, 2, D), 60), _rand((1, L, 2, D), 61)
    c = np.linspace(-3, 3, D).astype(np.float32)
    v = np.broadcast_to(c, (1, L, 2, D)).copy()
    o, _ = full_sequence_attention(q, k, v, g)
    np.testing.assert_allclose(o, np.broadcast_to(c, o.shape), rtol=0, atol=1e-5)


def test_zero_queries_give_mean_of_allowed_values():
    T, C, R, W = 3, 2, 1, 1
    g = ChunkGeometry(T, C, R, W)
    frames, D = 10, 8
    L = T * frames
    q = np.zeros((1, L, 1, D), np.float32)
    k, v = _rand((1, L, 1, D), 70), _rand((1, L, 1, D), 71)
    o, _ = full_sequence_attention(q, k, v, g, dtype=np.float64)
    # allowed keys of a query in chunk a: c_0 tokens [0, 3) and chunks a-1, a,
    # listed from the chunk boundaries (c_0 = 3 tokens, then chunks of 6).
    bounds = [0, 3] + list(range(9, L, 6)) + [L]
    bounds = sorted(set(bounds))
    chunks = [list(range(bounds[i], bounds[i + 1])) for i in range(len(bounds) - 1)]
    for a, toks in enumerate(chunks):
        keys = set(chunks[0])
        for c in (a - 1, a):
            if c >= 0:
                keys |= set(chunks[c])
        mean = v[0, sorted(keys), 0].astype(np.float64).mean(axis=0)
        for i in toks:
            np.testing.assert_allclose(o[0, i, 0], mean, rtol=0, atol=1e-12)


def test_output_rms_matches_random_logit_statistics():
    # unit-RMS q and k rows at D = 128 give logits ~ N(0, 1); then
    # E[RMS(O)] ~ sqrt(e / N) for N allowed keys of N(0, 1) values.
    w = WORKLOADS["wan14b_480p_chunk"]
    g = ChunkGeometry(w.tokens_per_frame, w.chunk_frames, w.ref_frames, w.window)
    rng = np.random.default_rng(5)
    n_keys, D = 4000, 128
    q = rng.standard_normal((1, 64, 1, D)).astype(np.float32)
    k = rng.standard_normal((1, n_keys, 1, D)).astype(np.float32)
    q /= np.sqrt((q * q).mean(-1, keepdims=True))
    k /= np.sqrt((k * k).mean(-1, keepdims=True))
    v = rng.standard_normal((1, n_keys, 1, D)).astype(np.float32)
    g_dense = ChunkGeometry(n_keys, 1, 1, 1)  # all keys in c_0
    o, _ = full_sequence_attention(q, k, v, g_dense)
    rms = float(np.sqrt(np.mean(o.astype(np.float64) ** 2)))
    assert abs(rms / math.sqrt(math.e / n_keys) - 1) < 0.1
    assert g.window == 1


# --------------------------------------------------------------------------- invariance


def test_disallowed_keys_have_no_influence_bitwise():
    T, C, R, W = 4, 2, 1, 1
    g = ChunkGeometry(T, C, R, W)
    L, D = T * 11, 16
    q, k, v = (_rand((1, L, 2, D), 80 + s) for s in range(3))
    q_chunk = 4
    q_rows = np.arange(chunk_start(q_chunk, g), chunk_start(q_chunk + 1, g))
    o_ref, lse_ref = full_sequence_attention(q, k, v, g, rows=q_rows)
    pos_chunk = chunk_of_frame(np.arange(L) // T, g)
    far = (pos_chunk >= 1) & (pos_chunk < q_chunk - W) | (pos_chunk > q_chunk)
    assert far.any()
    k2, v2 = k.copy(), v.copy()
    k2[0, far] = 3e4
    v2[0, far] = -7e4
    o2, lse2 = full_sequence_attention(q, k2, v2, g, rows=q_rows)
    assert np.array_equal(o_ref, o2) and np.array_equal(lse_ref, lse2)
    # ...while the previous chunk does matter
    prev = pos_chunk == q_chunk - 1
    k3 = k.copy()
    k3[0, prev] *= 2
    o3, _ = full_sequence_attention(q, k3, v, g, rows=q_rows)
    assert not np.allclose(o_ref, o3)


# --------------------------------------------------------------------------- streaming form


def test_streaming_history_equals_full_sequence_rows():
    w = WORKLOADS["tiny_f32"]
    g = ChunkGeometry(w.tokens_per_frame, w.chunk_frames, w.ref_frames, w.window)
    hist = StreamHistory(g)
    qs, ks, vs, outs = [], [], [], []
    for t in range(w.n_chunks + 1):
        d = draw_chunk(w, t)
        hist.append(t, d["k"], d["v"])
        o, _ = hist.attend(d["q"], t)
        qs.append(d["q"]); ks.append(d["k"]); vs.append(d["v"]); outs.append(o)
    q, k, v = (np.concatenate(x, axis=1) for x in (qs, ks, vs))
    o_full, _ = full_sequence_attention(q, k, v, g)
    np.testing.assert_allclose(np.concatenate(outs, axis=1), o_full, rtol=0, atol=1e-6)


def test_streaming_overwrite_replaces_latest_chunk():
    g = ChunkGeometry(2, 2, 1, 1)
    hist = StreamHistory(g)
    rng = np.random.default_rng(0)
    mk = lambda n: rng.standard_normal((1, n, 1, 8)).astype(np.float32)
    hist.append(0, mk(2), mk(2))
    hist.append(1, mk(4), mk(4))
    k_new, v_new = mk(4), mk(4)
    hist.append(1, k_new, v_new)
    _, k, v = hist.keys()
    assert np.array_equal(k[:, 2:], k_new) and np.array_equal(v[:, 2:], v_new)
    with pytest.raises(ValueError):
        hist.append(3, mk(4), mk(4))


def test_synthetic_inputs_are_bf16_exact_and_rms_normalised():
    w = WORKLOADS["wan14b_480p_chunk"]
    from synth.inputs import draw_tensor, bf16_bits_to_f32
    x, bits = draw_tensor((100, 4, 128), wid=w.wid, b=0, chunk=1, step=0, layer=0, tensor_id=1,
                          rms_normalise=True, dtype="bf16")
    assert np.array_equal(bf16_bits_to_f32(bits), x)
    rms = np.sqrt((x.astype(np.float64) ** 2).mean(-1))
    assert np.all(np.abs(rms - 1) < 1e-2)
    x2, _ = draw_tensor((100, 4, 128), wid=w.wid, b=0, chunk=1, step=0, layer=0, tensor_id=1,
                        rms_normalise=True, dtype="bf16")
    assert np.array_equal(x, x2)
    d = draw_qkv_sequence(WORKLOADS["tiny_f32"])
    assert d["q"].shape == (1, 9 * 64, 2, 64) and d["q"].dtype == np.float32


# --------------------------------------------------------------------------- fused K/V producer


def test_rms_normalise_rows_have_unit_rms_and_are_scale_free():
    from oracle import rms_normalise
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 17, 4, 128)) * rng.uniform(0.1, 10.0, size=(3, 17, 4, 1))
    y = rms_normalise(x)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=0, atol=1e-12)
    assert np.allclose(rms_normalise(7.5 * x), y, rtol=0, atol=1e-12)  # positive scale drops out
    assert np.array_equal(np.sign(y), np.sign(x))                      # direction kept per element


def test_rms_normalise_gain_and_eps_closed_forms():
    from oracle import rms_normalise
    x = np.full((1, 2, 3, 64), 2.0)                       # mean square 4
    g = np.arange(3 * 64, dtype=np.float64).reshape(3, 64)
    assert np.allclose(rms_normalise(x, g), g[None, None] * 1.0)             # 2 / sqrt(4) = 1
    assert np.allclose(rms_normalise(x, None, eps=5.0), 2.0 / 3.0)           # 2 / sqrt(4 + 5)
    one_hot = np.zeros((1, 1, 1, 128)); one_hot[..., 7] = 3.0                # mean square 9/128
    assert np.allclose(rms_normalise(one_hot)[..., 7], np.sqrt(128.0))


def test_rms_normalise_matches_torch_rms_norm():
    torch = pytest.importorskip("torch")
    from oracle import rms_normalise
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 9, 5, 128))
    g = rng.uniform(0.5, 1.5, size=(5, 128))
    for eps in (0.0, 1e-6):
        ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (128,), eps=eps).numpy() * g
        assert np.allclose(rms_normalise(x, g, eps), ref, rtol=1e-12, atol=1e-12)
