"""Host-side tests of the C ABI (no GPU needed).

The library must load and export every function ``include/tm.h`` declares;
argument validation must reject bad input on the host, before any launch,
with the documented status; the key-range planner's pair counts must equal
the oracle's mask counts.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import ChunkGeometry, allowed_mask
from oracle.attention import chunk_start

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tm.h")


@pytest.fixture(scope="module")
def tm():
    from paper_2506_03099_amd import tm as binding
    return binding


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tm_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_function(tm):
    names = _declared_functions()
    assert "tm_kv_append" in names and "tm_sparse_causal_attn_fwd" in names
    lib = tm.lib()
    for n in names:
        assert hasattr(lib, n), n


def _desc(tm, **kw):
    base = dict(batch=1, heads=40, head_dim=128, tokens_per_frame=1560, chunk_frames=3,
                ref_frames=1, window=1, dtype=tm.TM_BF16, softmax_scale=0.0)
    base.update(kw)
    return tm.tm_attn_desc(**base)


def test_cache_size_arithmetic(tm):
    # c_0 and each ring slot take their token count rounded up to 8; the total
    # is rounded up to the 64-token block of the V pool.
    d = _desc(tm)
    assert tm.tm_kv_cache_tokens(d) == 10944  # 1560 + 2 * 4680 = 10920 -> 171 blocks of 64
    assert tm.tm_kv_cache_bytes(d) == 40 * 10944 * 128 * 2
    d2 = _desc(tm, batch=2, tokens_per_frame=3600, dtype=tm.TM_F32, window=3)
    assert tm.tm_kv_cache_tokens(d2) == 46848  # 3600 + 4 * 10800 = 46800 -> 732 blocks
    assert tm.tm_kv_cache_bytes(d2) == 2 * 40 * 46848 * 128 * 4
    d3 = _desc(tm, tokens_per_frame=5, chunk_frames=3, ref_frames=1, window=2)
    assert tm.tm_kv_cache_tokens(d3) == 64  # 8 + 3 * 16 = 56 -> one block
    d4 = _desc(tm, tokens_per_frame=7, chunk_frames=10, ref_frames=3, window=12)
    assert tm.tm_kv_cache_tokens(d4) == 960  # 24 + 13 * 72 = 960


@pytest.mark.parametrize("kw", [dict(head_dim=96), dict(head_dim=0), dict(batch=0),
                                dict(heads=0), dict(tokens_per_frame=0), dict(chunk_frames=0),
                                dict(ref_frames=0), dict(window=-1), dict(window=13),
                                dict(dtype=7)])
def test_invalid_descriptor_has_no_cache_size(tm, kw):
    assert tm.tm_kv_cache_bytes(_desc(tm, **kw)) == 0
    assert tm.tm_kv_cache_tokens(_desc(tm, **kw)) == 0


FAKE = 1 << 40  # aligned, non-null, but not device memory


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), -2), (dict(dtype=5), -3), (dict(window=13), -2),
    (dict(softmax_scale=float("nan")), -1), (dict(softmax_scale=float("inf")), -1),
])
def test_forward_rejects_bad_descriptor(tm, kw, status):
    d = _desc(tm, **kw)
    st = tm.lib().tm_sparse_causal_attn_fwd(ctypes.byref(d), FAKE, -1, None, FAKE, FAKE, 21,
                                            FAKE, None, None)
    assert st == status
    assert tm.tm_last_error() != ""


def test_forward_rejects_bad_sequence_arguments(tm):
    d = _desc(tm)
    L = tm.lib()
    call = lambda qc, nf, q=FAKE, k=FAKE, v=FAKE, o=FAKE: L.tm_sparse_causal_attn_fwd(
        ctypes.byref(d), q, qc, None, k, v, nf, o, None, None)
    assert call(-1, 0) == tm.TM_E_SHAPE           # no frames
    assert call(8, 21) == tm.TM_E_SHAPE           # only chunks 0..7 exist
    assert call(-2, 21) == tm.TM_E_SHAPE
    assert call(-1, 21, q=None) == tm.TM_E_ARG     # NULL pointer
    assert call(-1, 21, k=FAKE + 8) == tm.TM_E_ARG  # misaligned
    assert call(-1, 21) == tm.TM_E_ARG             # not device memory


def test_append_and_cache_reject_bad_arguments(tm):
    L = tm.lib()
    d = _desc(tm)
    assert L.tm_kv_append(None, 0, FAKE, FAKE, 10, None) == tm.TM_E_ARG
    h = ctypes.c_void_p()
    assert L.tm_kv_cache_create(ctypes.byref(d), FAKE, FAKE, ctypes.byref(h)) == tm.TM_E_ARG
    assert L.tm_kv_cache_create(ctypes.byref(d), FAKE, FAKE + (1 << 32), ctypes.byref(h)) == tm.TM_E_ARG
    assert h.value is None
    assert L.tm_kv_cache_create(None, FAKE, FAKE, ctypes.byref(h)) == tm.TM_E_ARG
    assert L.tm_kv_cache_reset(None) == tm.TM_E_ARG
    assert L.tm_kv_cache_latest(None) == -1
    # the fused producer: no cache, or no queries
    assert L.tm_qkv_produce(None, 0, FAKE, FAKE, FAKE, None, None, 0.0, FAKE, 10, None) == tm.TM_E_ARG
    assert L.tm_qkv_produce(None, 0, None, FAKE, FAKE, None, None, 0.0, FAKE, 10, None) == tm.TM_E_ARG
    assert "q is NULL" in tm.tm_last_error()


def _oracle_pairs(n_frames, T, C, R, W, q_chunk):
    g = ChunkGeometry(T, C, R, W)
    L = n_frames * T
    pos = np.arange(L)
    if q_chunk >= 0:
        lo = chunk_start(q_chunk, g)
        hi = min(chunk_start(q_chunk + 1, g), L)
        qpos = pos[lo:hi]
    else:
        qpos = pos
    return int(allowed_mask(qpos, pos, g).sum())


@pytest.mark.parametrize("n_frames,T,C,R,W", [
    (21, 1560, 3, 1, 1), (21, 1560, 3, 3, 1), (9, 64, 2, 1, 1), (13, 7, 2, 1, 0),
    (13, 7, 2, 2, 3), (5, 11, 4, 1, 1), (2, 5, 3, 3, 1), (30, 3, 1, 1, 12),
])
def test_planner_pair_counts_equal_oracle_mask_counts(tm, n_frames, T, C, R, W):
    d = _desc(tm, heads=1, tokens_per_frame=T, chunk_frames=C, ref_frames=R, window=W)
    L = n_frames * T
    n_chunks = 1 if L <= R * T else 1 + -(-(L - R * T) // (C * T))
    if L <= 3000:
        assert tm.tm_allowed_pairs(d, -1, None, n_frames) == _oracle_pairs(n_frames, T, C, R, W, -1)
    for a in range(n_chunks):
        if L <= 3000 or a in (0, 1, n_chunks - 1):
            assert tm.tm_allowed_pairs(d, a, None, n_frames) == _oracle_pairs(n_frames, T, C, R, W, a)
    assert tm.tm_allowed_pairs(d, n_chunks, None, n_frames) == -1


def test_planner_full_sequence_480p_total(tm):
    d = _desc(tm)
    assert tm.tm_allowed_pairs(d, -1, None, 21) == 316_368_000


# --------------------------------------------------------------------------- audio cross-attention


def _adesc(tm, **kw):
    base = dict(batch=1, heads=40, head_dim=128, tokens_per_frame=1560, audio_per_frame=32,
                audio_frames=21, streams=1, half_window=2, dtype=tm.TM_BF16, softmax_scale=0.0)
    base.update(kw)
    return tm.tm_audio_desc(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=0), -3), (dict(dtype=9), -3), (dict(head_dim=96), -2), (dict(batch=0), -2),
    (dict(heads=0), -2), (dict(tokens_per_frame=0), -2), (dict(audio_per_frame=0), -2),
    (dict(audio_frames=0), -2), (dict(streams=0), -2), (dict(streams=33), -2),
    (dict(half_window=-1), -2), (dict(softmax_scale=float("nan")), -1),
    # windows that do not fit one workgroup's LDS: 5 * 58 = 290 > 288 keys at D = 128
    (dict(audio_per_frame=58), -2), (dict(head_dim=64, audio_per_frame=122), -2),
])
def test_audio_rejects_bad_descriptor(tm, kw, status):
    d = _adesc(tm, **kw)
    st = tm.lib().tm_audio_cross_attn_fwd(ctypes.byref(d), FAKE, 0, 4680, FAKE, FAKE, FAKE, FAKE, None)
    assert st == status, tm.tm_last_error()
    assert tm.tm_last_error() != ""


def test_audio_rejects_bad_arguments(tm):
    L = tm.lib()
    d = _adesc(tm)
    call = lambda ff, n, q=FAKE, ak=FAKE, av=FAKE, face=FAKE, o=FAKE: L.tm_audio_cross_attn_fwd(
        ctypes.byref(d), q, ff, n, ak, av, face, o, None)
    assert L.tm_audio_cross_attn_fwd(None, FAKE, 0, 10, FAKE, FAKE, FAKE, FAKE, None) == tm.TM_E_ARG
    assert call(0, 0) == tm.TM_OK                    # nothing to attend: no launch, no checks
    assert call(-1, 10) == tm.TM_E_SHAPE
    assert call(0, -1) == tm.TM_E_SHAPE
    assert call(19, 3 * 1560) == tm.TM_E_SHAPE       # frames 19..21, audio covers 0..20
    assert call(18, 3 * 1560 + 1) == tm.TM_E_SHAPE   # a 4th, partial frame: 18..21
    assert call(18, 3 * 1560, q=None) == tm.TM_E_ARG
    assert call(18, 3 * 1560, face=FAKE + 2) == tm.TM_E_ARG   # misaligned
    assert call(18, 3 * 1560) == tm.TM_E_ARG          # not device memory
    # the widest window fits: 288 keys at D = 128 (A = 57, w = 2: 285 keys)
    ok = _adesc(tm, audio_per_frame=57)
    st = L.tm_audio_cross_attn_fwd(ctypes.byref(ok), FAKE, 0, 10, FAKE, FAKE, FAKE, FAKE, None)
    assert st == tm.TM_E_ARG  # passes the shape checks, fails on the fake pointers
    # near the ends of the audio the window is clipped, so a wider A can fit there
    edge = _adesc(tm, audio_per_frame=90, audio_frames=3)  # frames 0..2: at most 3 * 90 = 270 keys
    st = L.tm_audio_cross_attn_fwd(ctypes.byref(edge), FAKE, 0, 1560, FAKE, FAKE, FAKE, FAKE, None)
    assert st == tm.TM_E_ARG


# --------------------------------------------------------------------------- backward


def test_backward_rejects_bad_arguments(tm):
    L = tm.lib()
    d = _desc(tm)
    call = lambda desc, nf, q=FAKE, lse=FAKE: L.tm_sparse_causal_attn_bwd(
        ctypes.byref(desc), nf, q, FAKE, FAKE, FAKE, lse, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert call(_desc(tm, dtype=tm.TM_F32), 21) == tm.TM_E_DTYPE
    assert call(_desc(tm, head_dim=96), 21) == tm.TM_E_SHAPE
    assert call(d, 0) == tm.TM_E_SHAPE
    assert call(d, 21, q=None) == tm.TM_E_ARG
    assert call(d, 21, lse=FAKE + 2) == tm.TM_E_ARG   # misaligned
    assert call(d, 21) == tm.TM_E_ARG                 # not device memory
    assert L.tm_sparse_causal_attn_bwd(None, 21, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                       FAKE, None) == tm.TM_E_ARG
