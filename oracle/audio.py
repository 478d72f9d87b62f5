"""Oracle of the audio cross-attention with a local window and a face mask
(test infrastructure only; never imported by the product path).

Paper: TalkingMachines, Sec. 4.1. The DiT's cross-attention layers gain keys
and values computed from audio tokens, and the tokens of each latent frame
cross-attend to them ("Audio Cross Attention with Attention Mask"); a local
mask restricts that attention to the face region; each latent frame sees only
the audio tokens of the five latent frames centred on it ("Audio Projection
Layer"); with several faces, each face takes its own audio stream, a silent
face a special (e.g. zero) embedding ("Speaking/Silence Mode").

Readings (the paper gives no formula):
* audio tokens are aligned to latent frames, ``A`` per frame: audio token j
  belongs to latent frame j // A; the audio covers frames 0 .. F_a - 1;
* the window of latent frame f is frames f - w .. f + w (w = 2 for five
  frames), clipped to 0 .. F_a - 1;
* the face mask acts on the query side: a query token with face id -1 (no
  face) receives no audio, its output is zero; a token of face m attends to
  audio stream m only (a silent face's stream holds the special embedding's
  keys and values: data, not a different computation);
* inside the window the attention is exact, softmax(scale * q K^T) V with
  scale = 1/sqrt(head_dim) unless given.

The definition is written out per query row: build that row's key list,
take the softmax, multiply by V. No tiling and no online softmax.
"""
from __future__ import annotations

import numpy as np


def audio_window(frame: int, audio_per_frame: int, audio_frames: int, half_window: int):
    """Audio token indices [lo, hi) that latent frame ``frame`` attends to."""
    f_lo = max(0, frame - half_window)
    f_hi = min(audio_frames - 1, frame + half_window)
    if f_lo > f_hi:
        raise ValueError("the frame's audio window is empty")
    return f_lo * audio_per_frame, (f_hi + 1) * audio_per_frame


def audio_cross_attention(q, ak, av, face, *, tokens_per_frame: int, audio_per_frame: int,
                          first_frame: int = 0, half_window: int = 2, scale=None,
                          heads=None, rows=None, dtype=np.float32):
    """Audio cross-attention of a run of latent-frame tokens.

    q: [B, n, H, D], row i in latent frame first_frame + i // tokens_per_frame;
    ak, av: [B, M, F_a * A, H, D], audio keys and values of M streams;
    face: [B, n] int, the stream each query token attends to, or -1 (none).
    ``heads`` / ``rows`` optionally select a subset (sampled comparisons).
    Returns o [B, n_rows, n_heads, D] in ``dtype``.
    """
    q = np.asarray(q)
    ak = np.asarray(ak)
    av = np.asarray(av)
    face = np.asarray(face)
    B, n, H, D = q.shape
    M, La = ak.shape[1], ak.shape[2]
    if La % audio_per_frame != 0:
        raise ValueError("audio length is not a whole number of frames")
    audio_frames = La // audio_per_frame
    if scale is None:
        scale = 1.0 / float(np.sqrt(D))
    heads = list(range(H)) if heads is None else list(heads)
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    o = np.zeros((B, len(rows), len(heads), D), dtype=dtype)
    for b in range(B):
        for ri, i in enumerate(rows):
            m = int(face[b, i])
            if m < 0:
                continue  # no face: no audio reaches this token
            if m >= M:
                raise ValueError("face id beyond the audio streams")
            f = first_frame + int(i) // tokens_per_frame
            lo, hi = audio_window(f, audio_per_frame, audio_frames, half_window)
            for hi_, h in enumerate(heads):
                qi = q[b, i, h, :].astype(dtype)
                kk = ak[b, m, lo:hi, h, :].astype(dtype)
                vv = av[b, m, lo:hi, h, :].astype(dtype)
                s = (kk @ qi) * dtype(scale)
                e = np.exp(s - s.max())
                p = e / e.sum()
                o[b, ri, hi_, :] = p @ vv
    return o
