"""Pins of the audio cross-attention oracle (``oracle.audio``).

The paper prints no numbers for it, so the oracle is pinned by: the window
pattern written by hand from Sec. 4.1 (golden file); PyTorch's CPU
scaled_dot_product_attention with an explicit boolean mask built from the
frame distance (a second construction of the key set), per stream, for the
general case, and without a mask where the window covers all audio; constant-V
and zero-Q closed forms; invariance to audio outside every window and to
streams no face uses. Planted mistakes in the oracle must fail a pin.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle.audio as aud

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_window(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([c == "1" for c in line])
    return np.array(rows, dtype=bool)


def _case(seed, B=2, M=3, T=5, A=3, Fa=7, frames=4, H=2, D=16, face_p=(0.3, 0.3, 0.2, 0.2)):
    rng = np.random.default_rng(seed)
    n = T * frames
    q = rng.standard_normal((B, n, H, D)).astype(np.float32)
    ak = rng.standard_normal((B, M, Fa * A, H, D)).astype(np.float32)
    av = rng.standard_normal((B, M, Fa * A, H, D)).astype(np.float32)
    face = rng.choice(np.arange(-1, M), size=(B, n), p=face_p[:M + 1] if len(face_p) == M + 1 else None)
    return q, ak, av, face


def _sdpa_reference(q, ak, av, face, T, A, first_frame, w):
    """Per stream: SDPA over every query row with mask |frame(q) - frame(k)| <= w;
    then each row keeps its own stream's result (zero for no face)."""
    B, n, H, D = q.shape
    M, La = ak.shape[1], ak.shape[2]
    fq = first_frame + np.arange(n) // T
    fk = np.arange(La) // A
    mask = torch.from_numpy(np.abs(fq[:, None] - fk[None, :]) <= w)
    out = np.zeros_like(q, dtype=np.float64)
    for b in range(B):
        for m in range(M):
            qt = torch.from_numpy(q[b].astype(np.float64)).permute(1, 0, 2)    # [H, n, D]
            kt = torch.from_numpy(ak[b, m].astype(np.float64)).permute(1, 0, 2)
            vt = torch.from_numpy(av[b, m].astype(np.float64)).permute(1, 0, 2)
            o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
            sel = face[b] == m
            out[b, sel] = o.permute(1, 0, 2).numpy()[sel]
    return out


def test_window_matches_golden_pattern():
    g = _golden_window("audio_window_fa7_w2.txt")
    for f in range(7):
        for A in (1, 4):
            lo, hi = aud.audio_window(f, A, 7, 2)
            got = np.zeros(7, dtype=bool)
            got[lo // A:hi // A] = True
            assert lo % A == 0 and hi % A == 0
            assert np.array_equal(got, g[f]), f


def test_general_case_matches_sdpa_with_frame_distance_mask():
    for seed, first in ((1, 0), (2, 3)):
        q, ak, av, face = _case(seed)
        o = aud.audio_cross_attention(q, ak, av, face, tokens_per_frame=5, audio_per_frame=3,
                                      first_frame=first, dtype=np.float64)
        ref = _sdpa_reference(q, ak, av, face, 5, 3, first, 2)
        assert np.allclose(o, ref, rtol=1e-10, atol=1e-12)
        assert np.all(o[face == -1] == 0)


def test_whole_audio_window_is_dense_cross_attention():
    q, ak, av, _ = _case(3, M=1)
    face = np.zeros(q.shape[:2], dtype=np.int64)
    o = aud.audio_cross_attention(q, ak, av, face, tokens_per_frame=5, audio_per_frame=3,
                                  half_window=10, dtype=np.float64)
    for b in range(q.shape[0]):
        qt = torch.from_numpy(q[b].astype(np.float64)).permute(1, 0, 2)
        kt = torch.from_numpy(ak[b, 0].astype(np.float64)).permute(1, 0, 2)
        vt = torch.from_numpy(av[b, 0].astype(np.float64)).permute(1, 0, 2)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt).permute(1, 0, 2).numpy()
        assert np.allclose(o[b], ref, rtol=1e-10, atol=1e-12)


def test_constant_values_and_zero_queries():
    q, ak, av, face = _case(4)
    B, M = ak.shape[:2]
    c = np.arange(1, M + 1, dtype=np.float32)[None, :, None, None, None] * np.ones_like(av)
    o = aud.audio_cross_attention(q, ak, c, face, tokens_per_frame=5, audio_per_frame=3,
                                  dtype=np.float64)
    want = np.where(face[..., None, None] >= 0, face[..., None, None] + 1.0, 0.0)
    assert np.allclose(o, np.broadcast_to(want, o.shape), rtol=0, atol=1e-12)
    # q = 0: the plain mean of the window's values (window from the frame distance)
    z = aud.audio_cross_attention(np.zeros_like(q), ak, av, face, tokens_per_frame=5,
                                  audio_per_frame=3, first_frame=1, dtype=np.float64)
    fk = np.arange(ak.shape[2]) // 3
    for b in range(B):
        for i in range(q.shape[1]):
            m = face[b, i]
            if m < 0:
                assert np.all(z[b, i] == 0)
                continue
            sel = np.abs(fk - (1 + i // 5)) <= 2
            assert np.allclose(z[b, i], av[b, m, sel].astype(np.float64).mean(0), atol=1e-12)


def test_audio_outside_every_window_and_unused_streams_do_not_matter():
    q, ak, av, face = _case(5, Fa=12, frames=3)
    face = np.where(face == 2, 1, face)  # stream 2 unused
    o = aud.audio_cross_attention(q, ak, av, face, tokens_per_frame=5, audio_per_frame=3)
    ak2, av2 = ak.copy(), av.copy()
    ak2[:, :, 5 * 3:] = 1e4   # frames 5.. lie outside the windows of frames 0..2
    av2[:, :, 5 * 3:] = -1e4
    ak2[:, 2] = 3e4
    av2[:, 2] = 7e4
    o2 = aud.audio_cross_attention(q, ak2, av2, face, tokens_per_frame=5, audio_per_frame=3)
    assert np.array_equal(o, o2)


def test_output_rms_of_random_logits():
    # unit-RMS q and k rows: logits ~ N(0, 1), so RMS(o) ~ sqrt(e / n_keys)
    rng = np.random.default_rng(6)
    A, D = 32, 128
    q = rng.standard_normal((1, 64, 2, D))
    ak = rng.standard_normal((1, 1, 9 * A, 2, D))
    av = rng.standard_normal((1, 1, 9 * A, 2, D))
    q /= np.sqrt((q * q).mean(-1, keepdims=True))
    ak /= np.sqrt((ak * ak).mean(-1, keepdims=True))
    face = np.zeros((1, 64), dtype=np.int64)
    o = aud.audio_cross_attention(q, ak, av, face, tokens_per_frame=16, audio_per_frame=A,
                                  first_frame=4, dtype=np.float64)   # frames 4..7: 5 full frames
    rms = float(np.sqrt(np.mean(o ** 2)))
    assert abs(rms / math.sqrt(math.e / (5 * A)) - 1) < 0.1


# --------------------------------------------------------------------------- planted mistakes


def _window_too_wide(frame, A, Fa, w):
    return aud.__dict__["_orig_window"](frame, A, Fa, w + 1)


def _window_unclipped_low(frame, A, Fa, w):
    lo, hi = aud.__dict__["_orig_window"](frame, A, Fa, w)
    return max(0, (frame - w) * A + A), hi


def _pins_hold():
    try:
        test_window_matches_golden_pattern()
        test_general_case_matches_sdpa_with_frame_distance_mask()
        test_constant_values_and_zero_queries()
    except AssertionError:
        return False
    return True


def test_unmutated_audio_oracle_passes():
    assert _pins_hold()


@pytest.mark.parametrize("name", ["window_too_wide", "window_unclipped_low", "face_ignored",
                                  "frame_offset_ignored", "stream_zero_always"])
def test_audio_mutants_fail_a_pin(monkeypatch, name):
    orig_window, orig_attn = aud.audio_window, aud.audio_cross_attention
    monkeypatch.setitem(aud.__dict__, "_orig_window", orig_window)
    if name == "window_too_wide":
        monkeypatch.setattr(aud, "audio_window", _window_too_wide)
    elif name == "window_unclipped_low":
        monkeypatch.setattr(aud, "audio_window", _window_unclipped_low)
    elif name == "face_ignored":
        monkeypatch.setattr(aud, "audio_cross_attention",
                            lambda q, ak, av, face, **kw: orig_attn(q, ak, av, np.maximum(face, 0), **kw))
    elif name == "frame_offset_ignored":
        monkeypatch.setattr(aud, "audio_cross_attention",
                            lambda q, ak, av, face, first_frame=0, **kw: orig_attn(q, ak, av, face, **kw))
    elif name == "stream_zero_always":
        def zero_stream(q, ak, av, face, **kw):
            return orig_attn(q, ak[:, :1], av[:, :1], np.where(face >= 0, 0, -1), **kw)
        monkeypatch.setattr(aud, "audio_cross_attention", zero_stream)
    assert not _pins_hold()
