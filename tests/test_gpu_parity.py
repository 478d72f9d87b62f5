"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every case draws seeded inputs from ``synth``, runs the library's kernels on
the GPU and compares with the oracle on the same values:
max |gpu - oracle| <= 1e-4 x RMS(oracle) for fp32, <= 2e-2 x RMS for bf16.
For bf16 inputs the small cases run each call twice, with the bf16 output and
with the fp32 output of the same kernel: the fp32 output is held to the bar
and the bf16 output must be its nearest-even rounding, bit for bit (where a
query sees only tens to hundreds of keys, |o| reaches several times its RMS
and the rounding of the bf16 format alone comes close to the bar).
Small cases compare every element (sizes span several query and key tiles
with ragged tails); the full-size workloads (480p chunk, 480p full sequence,
720p with two streams) compare sampled heads and rows that the oracle
computes one by one. The KV append is checked bit for bit.
"""
import ctypes

import numpy as np
import pytest
import torch

from gpu_helpers import (LSE_ATOL, assert_close, assert_rounds_to, chunk_to_dev, from_dev,
                         sample_rows, say, to_dev)
from oracle import ChunkGeometry, StreamHistory, full_sequence_attention
from oracle.attention import chunk_start
from synth import WORKLOADS, draw_chunk, draw_qkv_sequence
from synth.inputs import Workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tm():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2506_03099_amd import tm as binding
    binding.lib()
    return binding


def _geom(w):
    return ChunkGeometry(w.tokens_per_frame, w.chunk_frames, w.ref_frames, w.window)


def _desc(tm, w):
    return tm.make_desc(w.batch, w.heads, w.head_dim, w.tokens_per_frame, w.chunk_frames,
                        w.ref_frames, w.window, w.dtype)


def _small(wid, name, dtype, B, H, D, T, C, R, W, frames=0, chunks=0):
    return Workload(wid, name, dtype, B, H, D, T, C, R, W, n_frames=frames, n_chunks=chunks)


def _fwd(tm, desc, dtype, *args, **kw):
    """(output, fp32 output of the same call for bf16 inputs, else None)."""
    o = tm.tm_sparse_causal_attn_fwd(desc, *args, **kw)
    if dtype != "bf16":
        return o, None
    kw.pop("lse", None)
    kw.pop("o", None)
    return o, tm.tm_sparse_causal_attn_fwd_f32out(desc, *args, **kw)


def _check(o, of, want, dtype, what):
    """fp32: o within 1e-4 x RMS. bf16: o equals the rounded fp32 output of
    the same call, and that fp32 output is within 2e-2 x RMS."""
    torch.cuda.synchronize()
    if of is None:
        assert_close(from_dev(o), want, dtype, what)
    else:
        assert_rounds_to(o, of, what)
        assert_close(from_dev(of), want, "bf16", what)


# --------------------------------------------------------------------------- KV append


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("W", [0, 1, 2])
def test_kv_append_ring_is_bitwise_and_evicts(tm, dtype, W):
    T, C, R, B, H, D = 5, 2, 2, 2, 3, 64
    say(f"kv_append ring: dtype={dtype} W={W}")
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype)
    cache = tm.KVCache(desc)
    ib = torch.int16 if dtype == "bf16" else torch.int32
    cache.k_pool.view(ib).fill_(0x1357)
    cache.v_pool.view(ib).fill_(0x2468)
    exp_k = cache.k_pool.view(ib).cpu().numpy().copy()
    exp_v = cache.v_pool.view(ib).cpu().numpy().copy()
    rng = np.random.default_rng(W)
    RT, CT = R * T, C * T
    # Documented layout: c_0 at row 0, ring slot s at row 16 + 16 * s (c_0 and
    # chunks of 10 tokens each take 16 rows); V element (row t, dim d) at
    # block t // 64, row d, column t % 64; the V columns from the chunk's end
    # to the next multiple of 8 are zeros.
    assert cache.capacity == 64 and exp_v.shape == (B, H, 1, D, 64)
    seq = [(0, RT), (1, CT), (1, CT), (2, CT), (3, 3), (4, CT), (5, 7), (6, 1)]
    history = {}
    for chunk, n in seq:
        k = torch.from_numpy(rng.standard_normal((B, n, H, D)).astype(np.float32)).to(
            torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()
        v = torch.from_numpy(rng.standard_normal((B, n, H, D)).astype(np.float32)).to(k.dtype).cuda()
        tm.tm_kv_append(cache, chunk, k, v)
        off = 0 if chunk == 0 else 16 + ((chunk - 1) % (W + 1)) * 16
        kh = k.view(ib).cpu().numpy()
        vh = v.view(ib).cpu().numpy()
        exp_k[:, :, off:off + n, :] = kh.transpose(0, 2, 1, 3)
        n8 = (n + 7) // 8 * 8
        exp_v[:, :, 0, :, off:off + n8] = 0
        exp_v[:, :, 0, :, off:off + n] = vh.transpose(0, 2, 3, 1)
        torch.cuda.synchronize()
        assert np.array_equal(cache.k_pool.view(ib).cpu().numpy(), exp_k)
        assert np.array_equal(cache.v_pool.view(ib).cpu().numpy(), exp_v)
        history[chunk] = n
        assert cache.latest() == chunk
        assert cache.locate(chunk) == (off, n)
        for old in range(1, chunk - W):
            with pytest.raises(tm.TMError) as e:
                cache.locate(old)
            assert e.value.status == tm.TM_E_ORDER
        assert cache.locate(0) == (0, RT)


# --------------------------------------------------------------------------- small, every element

SMALL = [
    # wid, name, dtype, B, H, D, T, C, R, W, frames
    (101, "ragged_d128", "bf16", 1, 2, 128, 50, 3, 3, 1, 13),
    (121, "ragged_d128_r1", "bf16", 1, 2, 128, 50, 3, 1, 1, 13),
    (122, "tiny_shape_r1_bf16", "bf16", 1, 2, 64, 64, 2, 1, 1, 9),
    (123, "no_window_r1_b2", "bf16", 2, 3, 128, 33, 2, 1, 0, 11),
    (124, "window2_d64_r1", "bf16", 1, 2, 64, 40, 1, 1, 2, 12),
    (126, "chunks_below_tile_r1", "bf16", 1, 2, 128, 7, 3, 1, 1, 13),
    (102, "tiny_shape_bf16", "bf16", 1, 2, 64, 64, 2, 2, 1, 9),
    (103, "no_window_b2", "bf16", 2, 3, 128, 33, 2, 4, 0, 11),
    (104, "window2_d64", "bf16", 1, 2, 64, 40, 1, 4, 2, 12),
    (105, "literal_r3", "bf16", 1, 1, 128, 100, 3, 3, 1, 9),
    (106, "chunks_below_tile", "bf16", 1, 2, 128, 7, 3, 20, 1, 30),
    (107, "token_chunks_w12", "bf16", 1, 1, 64, 1, 1, 128, 12, 200),
    (111, "ragged_d128_f32", "f32", 1, 2, 128, 50, 3, 1, 1, 9),
    (112, "tiny_shape_f32", "f32", 1, 2, 64, 64, 2, 1, 1, 9),
    (113, "no_window_b2_f32", "f32", 2, 3, 128, 33, 2, 2, 0, 11),
    (114, "window2_d64_f32", "f32", 1, 2, 64, 40, 1, 1, 2, 10),
    (116, "chunks_below_tile_f32", "f32", 1, 2, 128, 7, 3, 1, 1, 13),
    (117, "token_chunks_w12_f32", "f32", 1, 1, 64, 1, 1, 1, 12, 40),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[1] for c in SMALL])
def test_full_sequence_matches_oracle_every_element(tm, case):
    wid, name, dtype, B, H, D, T, C, R, W, frames = case
    say(f"full sequence {name}: B={B} H={H} D={D} T={T} C={C} R={R} W={W} frames={frames}")
    w = _small(wid, name, dtype, B, H, D, T, C, R, W, frames=frames)
    g = _geom(w)
    d = draw_qkv_sequence(w)
    q, k, v = chunk_to_dev(d, dtype)
    desc = _desc(tm, w)
    L = frames * T
    lse = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    o, of = _fwd(tm, desc, dtype, q, -1, k=k, v=v, n_frames=frames, lse=lse)
    o_ref, lse_ref = full_sequence_attention(d["q"], d["k"], d["v"], g)
    _check(o, of, o_ref, dtype, f"{name} o")
    np.testing.assert_allclose(from_dev(lse), lse_ref, rtol=0, atol=LSE_ATOL[dtype])
    # each chunk on its own (mode with explicit ranges)
    n_chunks = 1 + -(-(L - R * T) // (C * T)) if L > R * T else 1
    chunks = range(n_chunks) if n_chunks <= 12 else sorted({0, 1, 2, 3, n_chunks // 2, n_chunks - 2, n_chunks - 1})
    for a in chunks:
        lo, hi = chunk_start(a, g), min(chunk_start(a + 1, g), L)
        qa = q[:, lo:hi].contiguous()
        oa, ofa = _fwd(tm, desc, dtype, qa, a, k=k, v=v, n_frames=frames)
        _check(oa, ofa, o_ref[:, lo:hi], dtype, f"{name} chunk {a}")


def test_few_keys_bf16(tm):
    """Chunks of a few tokens (c_0 = 7 tokens, chunks of 21): outputs average
    only 7-49 values, so |o| reaches several times its RMS."""
    w = _small(108, "few_keys", "bf16", 1, 2, 128, 7, 3, 1, 1, frames=13)
    g = _geom(w)
    d = draw_qkv_sequence(w)
    q, k, v = chunk_to_dev(d, "bf16")
    o, of = _fwd(tm, _desc(tm, w), "bf16", q, -1, k=k, v=v, n_frames=w.n_frames)
    o_ref, _ = full_sequence_attention(d["q"], d["k"], d["v"], g)
    _check(o, of, o_ref, "bf16", "few keys")


STREAM = [
    (201, "stream_tiny_f32", "f32", 1, 2, 64, 64, 2, 1, 1),
    (202, "stream_ragged_bf16", "bf16", 1, 3, 128, 50, 3, 3, 1),
    (203, "stream_w2_bf16", "bf16", 2, 2, 64, 30, 2, 5, 2),
    (204, "stream_w0_f32", "f32", 1, 2, 128, 20, 3, 2, 0),
]


@pytest.mark.parametrize("case", STREAM, ids=[c[1] for c in STREAM])
def test_streaming_matches_oracle_history(tm, case):
    wid, name, dtype, B, H, D, T, C, R, W = case
    say(f"streaming {name}")
    w = _small(wid, name, dtype, B, H, D, T, C, R, W, chunks=6)
    g = _geom(w)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    # chunk 0, then 1..5 with an overwrite of chunk 3 and a partial last chunk
    plan = [(0, None, 0), (1, None, 0), (2, None, 0), (3, None, 0), (3, None, 1), (4, None, 0),
            (5, C * T - 7, 0)]
    for chunk, n, step in plan:
        dd = draw_chunk(w, chunk, n, step=step)
        q, k, v = chunk_to_dev(dd, dtype)
        tm.tm_kv_append(cache, chunk, k, v)
        hist.append(chunk, dd["k"], dd["v"])
        lse = torch.empty((B, H, q.shape[1]), dtype=torch.float32, device="cuda")
        o, of = _fwd(tm, desc, dtype, q, chunk, cache=cache, lse=lse)
        o_ref, lse_ref = hist.attend(dd["q"], chunk)
        _check(o, of, o_ref, dtype, f"{name} chunk {chunk} step {step}")
        np.testing.assert_allclose(from_dev(lse), lse_ref, rtol=0,
                                   atol=LSE_ATOL[dtype])


def test_tiny_f32_workload_streaming_and_full_sequence(tm):
    """The tiny fp32 workload: 4 chunks streamed after the reference, all heads,
    then the same 9 frames in the full-sequence form; both against the oracle."""
    w = WORKLOADS["tiny_f32"]
    g = _geom(w)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    qs, ks, vs = [], [], []
    for t in range(w.n_chunks + 1):
        dd = draw_chunk(w, t)
        q, k, v = chunk_to_dev(dd, "f32")
        tm.tm_kv_append(cache, t, k, v)
        hist.append(t, dd["k"], dd["v"])
        o = tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=cache)
        torch.cuda.synchronize()
        o_ref, _ = hist.attend(dd["q"], t)
        n_keys = tm.tm_allowed_pairs(desc, t, cache) // q.shape[1]
        say(f"tiny_f32 chunk {t}: {q.shape[1]} queries x {n_keys} keys")
        assert n_keys == (64 if t == 0 else 192 if t == 1 else 320)
        assert_close(from_dev(o), o_ref, "f32", f"tiny chunk {t}")
        qs.append(q); ks.append(k); vs.append(v)
    q, k, v = (torch.cat(x, dim=1).contiguous() for x in (qs, ks, vs))
    o = tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=w.n_frames)
    torch.cuda.synchronize()
    o_ref, _ = full_sequence_attention(from_dev(q), from_dev(k), from_dev(v), g)
    assert_close(from_dev(o), o_ref, "f32", "tiny full sequence")


# --------------------------------------------------------------------------- invariants on the GPU


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_disallowed_keys_are_never_read(tm, dtype):
    """NaN in every key/value a query chunk may not see changes nothing, bit for bit."""
    w = _small(301, "poison", dtype, 1, 2, 128, 50, 3, 1, 1, frames=16)
    g = _geom(w)
    d = draw_qkv_sequence(w)
    q, k, v = chunk_to_dev(d, dtype)
    desc = _desc(tm, w)
    L = w.n_frames * w.tokens_per_frame
    for a in (3, 5):
        lo, hi = chunk_start(a, g), min(chunk_start(a + 1, g), L)
        qa = q[:, lo:hi].contiguous()
        clean = tm.tm_sparse_causal_attn_fwd(desc, qa, a, k=k, v=v, n_frames=w.n_frames)
        kp, vp = k.clone(), v.clone()
        allowed = np.zeros(L, bool)
        allowed[:chunk_start(1, g)] = True
        allowed[chunk_start(a - 1, g):hi] = True
        bad = torch.from_numpy(~allowed).cuda()
        kp[:, bad] = float("nan")
        vp[:, bad] = float("nan")
        dirty = tm.tm_sparse_causal_attn_fwd(desc, qa, a, k=kp, v=vp, n_frames=w.n_frames)
        torch.cuda.synchronize()
        assert torch.equal(clean, dirty), f"chunk {a}"
        assert torch.isfinite(dirty.float()).all()


def test_unfilled_cache_rows_are_never_read(tm):
    w = _small(302, "poison_cache", "bf16", 1, 2, 128, 40, 3, 1, 1, chunks=3)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    cache.k_pool.fill_(float("nan"))
    cache.v_pool.fill_(float("nan"))
    for t, n in ((0, None), (1, 50), (2, 77)):  # partial chunks leave NaN rows behind
        dd = draw_chunk(w, t, n)
        q, k, v = chunk_to_dev(dd, "bf16")
        tm.tm_kv_append(cache, t, k, v)
        o = tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=cache)
        torch.cuda.synchronize()
        assert torch.isfinite(o.float()).all(), f"chunk {t}"


def test_repeatable_bitwise_and_output_canaries(tm):
    w = _small(303, "repeat", "bf16", 1, 4, 128, 90, 3, 1, 1, frames=10)
    d = draw_qkv_sequence(w)
    q, k, v = chunk_to_dev(d, "bf16")
    desc = _desc(tm, w)
    n = q.numel()
    buf = torch.full((n + 4096,), 7.0, dtype=torch.bfloat16, device="cuda")
    o = buf[2048:2048 + n].view(q.shape)
    tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=w.n_frames, o=o)
    first = o.clone()
    for _ in range(3):
        tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=w.n_frames, o=o)
        torch.cuda.synchronize()
        assert torch.equal(o, first)
    assert torch.all(buf[:2048] == 7.0) and torch.all(buf[2048 + n:] == 7.0)


@pytest.mark.parametrize("form", ["cache", "sequence"])
def test_first_call_equals_repeated_calls_480p(tm, form):
    """The first launch on freshly written K/V (cold caches, slow tile loads)
    must give bit for bit what repeated launches give: a tile read from LDS
    before its loads have landed would show up here."""
    w = WORKLOADS["wan14b_480p_stream"]
    desc = _desc(tm, w)
    say(f"first call vs repeated, 480p chunk 1, {form}")
    cache = tm.KVCache(desc) if form == "cache" else None
    ks, vs = [], []
    for t in range(2):
        q, k, v = chunk_to_dev(draw_chunk(w, t, step=1), "bf16")
        ks.append(k); vs.append(v)
        if cache is not None:
            tm.tm_kv_append(cache, t, k, v)
    if cache is not None:
        run = lambda: tm.tm_sparse_causal_attn_fwd(desc, q, 1, cache=cache)
    else:
        K, V = (torch.cat(x, dim=1).contiguous() for x in (ks, vs))
        frames = w.ref_frames + w.chunk_frames
        run = lambda: tm.tm_sparse_causal_attn_fwd(desc, q, 1, k=K, v=V, n_frames=frames)
    first = run()
    torch.cuda.synchronize()
    for _ in range(3):
        again = run()
        torch.cuda.synchronize()
        assert torch.equal(first, again)


def test_streaming_equals_full_sequence_on_gpu(tm):
    w = _small(304, "stream_vs_full", "bf16", 1, 2, 128, 60, 3, 3, 1, chunks=4)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    qs, ks, vs, outs = [], [], [], []
    for t in range(w.n_chunks + 1):
        dd = draw_chunk(w, t)
        q, k, v = chunk_to_dev(dd, "bf16")
        tm.tm_kv_append(cache, t, k, v)
        outs.append(tm.tm_sparse_causal_attn_fwd_f32out(desc, q, t, cache=cache))
        qs.append(q); ks.append(k); vs.append(v)
    q, k, v = (torch.cat(x, dim=1).contiguous() for x in (qs, ks, vs))
    frames = w.ref_frames + w.n_chunks * w.chunk_frames
    o_full = tm.tm_sparse_causal_attn_fwd_f32out(desc, q, -1, k=k, v=v, n_frames=frames)
    torch.cuda.synchronize()
    # the two forms visit the keys in different orders (ring slots vs sequence)
    assert_close(from_dev(torch.cat(outs, dim=1)), from_dev(o_full), "bf16", "stream vs full")


# --------------------------------------------------------------------------- GPU-side argument errors


def test_argument_errors_with_real_device_memory(tm):
    w = _small(305, "errors", "bf16", 1, 2, 64, 64, 2, 2, 1, chunks=3)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    d0 = draw_chunk(w, 0)
    q0, k0, v0 = chunk_to_dev(d0, "bf16")
    d1 = draw_chunk(w, 1)
    q1, k1, v1 = chunk_to_dev(d1, "bf16")

    def status(fn, *a, **kw):
        with pytest.raises(tm.TMError) as e:
            fn(*a, **kw)
        return e.value.status

    assert status(tm.tm_kv_append, cache, 1, k1, v1) == tm.TM_E_ORDER  # chunk 0 first
    assert status(tm.tm_sparse_causal_attn_fwd, desc, q0, 0, cache=cache) == tm.TM_E_ORDER
    tm.tm_kv_append(cache, 0, k0, v0)
    assert status(tm.tm_kv_append, cache, 2, k1, v1) == tm.TM_E_ORDER  # skips chunk 1
    big = torch.zeros((1, 2 * w.chunk_tokens, 2, 64), dtype=torch.bfloat16, device="cuda")
    assert status(tm.tm_kv_append, cache, 1, big, big) == tm.TM_E_CAPACITY
    tm.tm_kv_append(cache, 1, k1, v1)
    assert status(tm.tm_sparse_causal_attn_fwd, desc, q1, 0, cache=cache) == tm.TM_E_ORDER
    other = tm.make_desc(1, 2, 64, 64, 2, 2, 0, "bf16")
    assert status(tm.tm_sparse_causal_attn_fwd, other, q1, 1, cache=cache) == tm.TM_E_ARG
    assert status(tm.tm_sparse_causal_attn_fwd, desc, q1.cpu(), 1, cache=cache) == tm.TM_E_ARG
    # a pointer whose tensor would run past the end of its allocation
    hip = ctypes.CDLL("libamdhip64.so")
    base, size = ctypes.c_void_p(), ctypes.c_size_t()
    assert hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size),
                                     ctypes.c_void_p(q1.data_ptr())) == 0
    near_end = base.value + size.value - 64
    st = tm.lib().tm_sparse_causal_attn_fwd(ctypes.byref(desc), near_end, 1, cache.handle, None,
                                            None, 0, q1.data_ptr(), None, None)
    assert st == tm.TM_E_ARG
    # the failed calls changed nothing: chunk 1 still attends correctly
    o, of = _fwd(tm, desc, "bf16", q1, 1, cache=cache)
    hist = StreamHistory(_geom(w))
    hist.append(0, d0["k"], d0["v"])
    hist.append(1, d1["k"], d1["v"])
    _check(o, of, hist.attend(d1["q"], 1)[0], "bf16", "after errors")


# --------------------------------------------------------------------------- full-size workloads, sampled


def test_480p_chunk_sampled(tm):
    """WAN-14B 480p chunk: 4680 queries over 1560 ref + 4680 previous + 4680 current keys."""
    w = WORKLOADS["wan14b_480p_chunk"]
    g = _geom(w)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    for t in range(w.n_chunks + 1):
        dd = draw_chunk(w, t)
        q, k, v = chunk_to_dev(dd, "bf16")
        tm.tm_kv_append(cache, t, k, v)
        hist.append(t, dd["k"], dd["v"])
    lse = torch.empty((1, w.heads, q.shape[1]), dtype=torch.float32, device="cuda")
    o = tm.tm_sparse_causal_attn_fwd(desc, q, w.n_chunks, cache=cache, lse=lse)
    torch.cuda.synchronize()
    assert tm.tm_allowed_pairs(desc, w.n_chunks, cache) == 4680 * 10920
    heads = [0, 17, 39]
    rows = sample_rows(q.shape[1])
    say(f"480p chunk: comparing heads {heads}, {len(rows)} rows")
    o_ref, lse_ref = hist.attend(dd["q"], w.n_chunks, heads=heads, rows=rows)
    got = from_dev(o)[:, rows][:, :, heads]
    assert_close(got, o_ref, "bf16", "480p chunk")
    np.testing.assert_allclose(from_dev(lse)[:, heads][:, :, rows], lse_ref, rtol=0, atol=LSE_ATOL["bf16"])
    # output statistics over every head and row: RMS ~ sqrt(e / 10920)
    rms = float(torch.sqrt((o.float() ** 2).mean()))
    assert abs(rms / np.sqrt(np.e / 10920) - 1) < 0.1


def test_480p_full_sequence_sampled(tm):
    """21 latent frames x 1560 tokens in one call; rows sampled in every chunk."""
    w = WORKLOADS["wan14b_480p_full_sequence"]
    g = _geom(w)
    d = draw_qkv_sequence(w)
    q, k, v = chunk_to_dev(d, "bf16")
    desc = _desc(tm, w)
    o, of = _fwd(tm, desc, "bf16", q, -1, k=k, v=v, n_frames=w.n_frames)
    torch.cuda.synchronize()
    assert_rounds_to(o, of, "480p full sequence")
    L = w.n_frames * w.tokens_per_frame
    bounds = [chunk_start(a, g) for a in range(9)]
    rows = set(sample_rows(L, k=64).tolist())
    for b in bounds[1:]:
        if b < L:
            rows.update({b - 1, b})
    rows = np.array(sorted(rows))
    heads = [3, 29]
    say(f"480p full sequence: heads {heads}, {len(rows)} rows")
    o_ref, _ = full_sequence_attention(d["q"], d["k"], d["v"], g, heads=heads, rows=rows)
    # the kernel's arithmetic (fp32 output) against the RMS of every compared
    # row together (c_0's rows see 1560 keys and have about 2.6 times the
    # output scale of the rows that see 10920)
    assert_close(from_dev(of)[:, rows][:, :, heads], o_ref, "bf16", "480p full sequence (fp32 out)")
    # the bf16 output itself, each query chunk's rows against that chunk's RMS
    got = from_dev(o)[:, rows][:, :, heads]
    chunk_of_row = np.searchsorted(np.array(bounds[1:]), rows, side="right")
    for a in np.unique(chunk_of_row):
        sel = chunk_of_row == a
        assert_close(got[:, sel], o_ref[:, sel], "bf16", f"480p full sequence chunk {a}")


def test_720p_two_streams_sampled(tm):
    """720p chunk, batch of two independent streams: 10800 queries x 25200 keys each."""
    w = WORKLOADS["wan14b_720p_chunk_b2"]
    g = _geom(w)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    for t in range(w.n_chunks + 1):
        dd = draw_chunk(w, t)
        q, k, v = chunk_to_dev(dd, "bf16")
        tm.tm_kv_append(cache, t, k, v)
        hist.append(t, dd["k"], dd["v"])
        del k, v
    o = tm.tm_sparse_causal_attn_fwd(desc, q, w.n_chunks, cache=cache)
    torch.cuda.synchronize()
    heads = [5, 38]
    rows = sample_rows(q.shape[1], k=48)
    say(f"720p b2: heads {heads}, {len(rows)} rows, both streams")
    o_ref, _ = hist.attend(dd["q"], w.n_chunks, heads=heads, rows=rows)
    assert_close(from_dev(o)[:, rows][:, :, heads], o_ref, "bf16", "720p b2")


VARIANTS = ["paper_512_chunk", "paper_480p_chunk7", "paper_720x720_chunk", "window2_ref3_stream"]


@pytest.mark.parametrize("name", VARIANTS)
def test_paper_variants_streamed_sampled(tm, name):
    """Shapes the paper also reports (deployed 512x512 resolution, 7-frame
    chunks, 720x720 frames with token counts that are not multiples of 8, a
    window of two chunks with a three-frame c_0): streamed through the cache,
    sampled parity at every chunk from the first that sees the full window."""
    w = WORKLOADS[name]
    g = _geom(w)
    desc = _desc(tm, w)
    cache = tm.KVCache(desc)
    hist = StreamHistory(g)
    heads = [0, w.heads - 1]
    for t in range(w.n_chunks + 1):
        dd = draw_chunk(w, t)
        q, k, v = chunk_to_dev(dd, "bf16")
        tm.tm_kv_append(cache, t, k, v)
        hist.append(t, dd["k"], dd["v"])
        o = tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=cache)
        if t < min(w.window + 1, w.n_chunks):
            continue
        torch.cuda.synchronize()
        rows = sample_rows(q.shape[1], k=32)
        o_ref, _ = hist.attend(dd["q"], t, heads=heads, rows=rows)
        say(f"{name}: chunk {t}, {q.shape[1]} queries, heads {heads}, {len(rows)} rows")
        assert_close(from_dev(o)[:, rows][:, :, heads], o_ref, "bf16", f"{name} chunk {t}")


def test_480p_streaming_loop_two_steps_sampled(tm):
    """The streaming loop at 480p shapes: one cache per denoising step, chunks
    1..3 appended and attended at both steps; sampled parity per (chunk, step)."""
    w = WORKLOADS["wan14b_480p_stream"]
    g = _geom(w)
    desc = _desc(tm, w)
    caches = [tm.KVCache(desc) for _ in range(2)]
    hists = [StreamHistory(g) for _ in range(2)]
    heads, rows = [11], sample_rows(w.chunk_tokens, k=32)
    for t in range(4):
        for s in range(2):
            dd = draw_chunk(w, t, step=s)
            q, k, v = chunk_to_dev(dd, "bf16")
            tm.tm_kv_append(caches[s], t, k, v)
            hists[s].append(t, dd["k"], dd["v"])
            o = tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=caches[s])
            if t >= 1:
                torch.cuda.synchronize()
                o_ref, _ = hists[s].attend(dd["q"], t, heads=heads, rows=rows)
                assert_close(from_dev(o)[:, rows][:, :, heads], o_ref, "bf16",
                             f"480p stream chunk {t} step {s}")
