"""Seeded synthetic q/k/v generator and the named workload shapes.

Every tensor is drawn from ``numpy.random.default_rng`` keyed by a
``SeedSequence`` built from (base seed, workload id, batch index, chunk index,
denoising step, layer, tensor id), so any single chunk of any stream can be
regenerated on its own. Values are N(0, 1) in fp32; queries and keys are then
divided by their root-mean-square over the head dimension (one row per token
and head, no gain, no epsilon); for bfloat16 workloads every value is rounded
to nearest-even bfloat16 and handed out both as raw 16-bit patterns (for upload
to the device) and as the exactly equal fp32 values (for the CPU side).

Layout of every tensor: ``[n_tokens, heads, head_dim]`` for one batch element;
callers stack batch elements in front to get ``[B, L, H, D]``.

The latent shapes follow the WAN2.1-14B image-to-video backbone the paper
builds on (Sec. 4.1): 40 heads of width 128, a 16x spatial patch grid per
latent frame (480x832 -> 30x52 = 1560 tokens, 720x1280 -> 45x80 = 3600), and
the paper's chunking of the 21-latent-frame clip into chunks of 3 latent
frames (Sec. 4.2, chunked processing).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

TENSOR_Q, TENSOR_K, TENSOR_V = 0, 1, 2
FULL_SEQUENCE_CHUNK = 1000  # seed slot used when a whole sequence is drawn at once


@dataclass(frozen=True)
class Workload:
    """Shape of one synthetic workload.

    tokens_per_frame (T), chunk_frames (C), ref_frames (R) and window (W)
    describe the chunk geometry; ``n_frames`` is the sequence length in latent
    frames for the full-sequence form; ``n_chunks`` the number of streamed
    chunks for the streaming form.
    """

    wid: int
    name: str
    dtype: str  # "f32" or "bf16"
    batch: int
    heads: int
    head_dim: int
    tokens_per_frame: int
    chunk_frames: int
    ref_frames: int
    window: int
    n_frames: int = 0
    n_chunks: int = 0
    steps: int = 1
    layers: int = 1
    notes: str = field(default="", compare=False)

    @property
    def chunk_tokens(self) -> int:
        return self.chunk_frames * self.tokens_per_frame

    @property
    def ref_tokens(self) -> int:
        return self.ref_frames * self.tokens_per_frame


WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in [
        Workload(1, "tiny_f32", "f32", 1, 2, 64, 64, 2, 1, 1, n_frames=9, n_chunks=4,
                 notes="64 tokens/frame, chunk of 2 frames, 4 streamed chunks"),
        Workload(2, "wan14b_480p_chunk", "bf16", 1, 40, 128, 1560, 3, 1, 1, n_chunks=2,
                 notes="one 4680-query chunk over 1560 ref + 4680 previous + 4680 current keys"),
        Workload(3, "wan14b_480p_full_sequence", "bf16", 1, 40, 128, 1560, 3, 1, 1, n_frames=21,
                 notes="21 latent frames: reference frame + six 3-frame chunks + one 2-frame chunk"),
        Workload(4, "wan14b_480p_stream", "bf16", 1, 40, 128, 1560, 3, 1, 1, n_chunks=10,
                 steps=2, layers=40,
                 notes="10 chunks x 2 denoising steps x 40 layers of append + attention"),
        Workload(5, "wan14b_720p_chunk_b2", "bf16", 2, 40, 128, 3600, 3, 1, 1, n_chunks=2,
                 notes="two independent streams, one 10800-query chunk over 25200 keys each"),
        # Variants the paper reports (parity cases): its deployed 512x512
        # resolution (32x32 patches per latent frame), 7-frame chunks, a
        # 720x720 frame (45x45 patches), and a window of two previous chunks
        # with a three-frame c_0. The last three use 8 heads to keep the
        # oracle's share of the test time small; heads are independent.
        Workload(6, "paper_512_chunk", "bf16", 1, 40, 128, 1024, 3, 1, 1, n_chunks=2,
                 notes="3072 queries over 1024 ref + 3072 previous + 3072 current keys"),
        Workload(7, "paper_480p_chunk7", "bf16", 1, 8, 128, 1560, 7, 1, 1, n_chunks=2,
                 notes="7-frame chunks: 10920 queries over 1560 + 10920 + 10920 keys"),
        Workload(8, "paper_720x720_chunk", "bf16", 1, 8, 128, 2025, 3, 1, 1, n_chunks=2,
                 notes="6075 queries over 2025 + 6075 + 6075 keys (token counts not multiples of 8)"),
        Workload(9, "window2_ref3_stream", "bf16", 1, 8, 128, 1560, 3, 3, 2, n_chunks=4,
                 notes="W = 2 and a 3-frame c_0: chunks 3 and 4 see c_0 + three chunks"),
    ]
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bfloat16, nearest-even, returning the 16-bit patterns.

    Finite inputs only (the generator never produces inf/NaN).
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    rounded = u + np.uint32(0x7FFF) + lsb
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to fp32."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(wid: int, b: int, chunk: int, step: int, layer: int, tensor_id: int,
         base_seed: int = 0) -> np.random.Generator:
    return np.random.default_rng(
        np.random.SeedSequence([base_seed, wid, b, chunk, step, layer, tensor_id]))


def draw_tensor(shape, *, wid: int, b: int, chunk: int, step: int, layer: int,
                tensor_id: int, rms_normalise: bool, dtype: str, base_seed: int = 0):
    """Draw one seeded tensor of ``shape`` (last axis = head_dim).

    Returns ``(f32_values, bf16_bits_or_None)``. For ``dtype == "bf16"`` the
    fp32 array holds exactly the bfloat16 values whose bit patterns are
    returned alongside.
    """
    x = _rng(wid, b, chunk, step, layer, tensor_id, base_seed).standard_normal(
        size=shape, dtype=np.float32)
    if rms_normalise:
        x /= np.sqrt(np.mean(x * x, axis=-1, keepdims=True, dtype=np.float32))
    if dtype == "f32":
        return x, None
    if dtype != "bf16":
        raise ValueError(f"unknown dtype {dtype!r}")
    bits = f32_to_bf16_bits(x)
    return bf16_bits_to_f32(bits), bits


def _draw_qkv(n_tok: int, w: Workload, b: int, chunk: int, step: int, layer: int,
              base_seed: int):
    shape = (n_tok, w.heads, w.head_dim)
    out = []
    for tid in (TENSOR_Q, TENSOR_K, TENSOR_V):
        out.append(draw_tensor(shape, wid=w.wid, b=b, chunk=chunk, step=step, layer=layer,
                               tensor_id=tid, rms_normalise=tid != TENSOR_V, dtype=w.dtype,
                               base_seed=base_seed))
    return out


def draw_chunk(w: Workload, chunk: int, n_tok: int | None = None, *, step: int = 0,
               layer: int = 0, base_seed: int = 0):
    """q, k, v for one chunk of every batch element, shaped ``[B, n_tok, H, D]``.

    ``chunk == 0`` is the reference chunk (``R*T`` tokens by default), later
    chunks hold ``C*T`` tokens unless ``n_tok`` says otherwise.
    Returns a dict with fp32 arrays ``q, k, v`` and, for bf16 workloads, the
    bit patterns ``q_bits, k_bits, v_bits`` (uint16).
    """
    if n_tok is None:
        n_tok = w.ref_tokens if chunk == 0 else w.chunk_tokens
    per_b = [_draw_qkv(n_tok, w, b, chunk, step, layer, base_seed) for b in range(w.batch)]
    res = {}
    for i, name in enumerate("qkv"):
        res[name] = np.stack([pb[i][0] for pb in per_b])
        if w.dtype == "bf16":
            res[name + "_bits"] = np.stack([pb[i][1] for pb in per_b])
    return res


def draw_qkv_sequence(w: Workload, n_frames: int | None = None, *, step: int = 0,
                      layer: int = 0, base_seed: int = 0):
    """q, k, v for a whole ``n_frames``-frame sequence, shaped ``[B, L, H, D]``."""
    if n_frames is None:
        n_frames = w.n_frames
    n_tok = n_frames * w.tokens_per_frame
    per_b = [_draw_qkv(n_tok, w, b, FULL_SEQUENCE_CHUNK, step, layer, base_seed)
             for b in range(w.batch)]
    res = {}
    for i, name in enumerate("qkv"):
        res[name] = np.stack([pb[i][0] for pb in per_b])
        if w.dtype == "bf16":
            res[name + "_bits"] = np.stack([pb[i][1] for pb in per_b])
    return res


# --------------------------------------------------------------------------- audio cross-attention


@dataclass(frozen=True)
class AudioWorkload:
    """Shape of one synthetic audio cross-attention workload.

    The query rows are ``n_frames`` latent frames of a ``grid_h x grid_w``
    patch grid starting at latent frame ``first_frame``; the audio holds
    ``audio_per_frame`` tokens per latent frame for ``audio_frames`` frames and
    ``streams`` faces; ``half_window`` frames on each side (2: five frames).
    """

    wid: int
    name: str
    batch: int
    heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    audio_per_frame: int
    audio_frames: int
    streams: int
    half_window: int
    first_frame: int
    n_frames: int
    notes: str = field(default="", compare=False)

    @property
    def tokens_per_frame(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def n_tok(self) -> int:
        return self.n_frames * self.tokens_per_frame


AUDIO_WORKLOADS: dict[str, AudioWorkload] = {
    w.name: w
    for w in [
        AudioWorkload(20, "wan14b_480p_audio_chunk", 1, 40, 128, 30, 52, 32, 21, 1, 2, 4, 3,
                      notes="one 3-frame chunk (frames 4..6 of 21) of 1560 tokens per frame, "
                            "one face, 32 audio tokens per latent frame, five-frame window"),
        AudioWorkload(21, "wan14b_480p_audio_2faces", 1, 8, 128, 30, 52, 32, 21, 2, 2, 18, 3,
                      notes="the last chunk (frames 18..20, windows clipped), two faces"),
    ]
}


def face_ids(grid_h: int, grid_w: int, n_frames: int, streams: int, batch: int = 1):
    """Face id of every token, int32 ``[batch, n_frames * grid_h * grid_w]``:
    ``streams`` elliptical face regions side by side in the upper half of
    every frame (face m centred at column (m + 1) / (streams + 1) of the
    width, row 0.4 of the height; semi-axes 0.4 / (streams + 1) of the width
    and 0.22 of the height), -1 elsewhere."""
    y, x = np.meshgrid(np.arange(grid_h) + 0.5, np.arange(grid_w) + 0.5, indexing="ij")
    ids = np.full((grid_h, grid_w), -1, dtype=np.int32)
    ry = 0.22 * grid_h
    rx = 0.4 * grid_w / (streams + 1)
    for m in range(streams):
        cx = grid_w * (m + 1) / (streams + 1)
        cy = 0.4 * grid_h
        ids[((x - cx) / rx) ** 2 + ((y - cy) / ry) ** 2 <= 1.0] = m
    frame = ids.reshape(-1)
    return np.broadcast_to(np.tile(frame, n_frames), (batch, n_frames * frame.size)).copy()


def draw_audio(w: AudioWorkload, *, layer: int = 0, base_seed: int = 0):
    """Seeded bf16 inputs of an audio workload.

    q ``[B, n_tok, H, D]`` and the audio keys ``ak`` ``[B, M, F_a * A, H, D]``
    are RMS-normalised per (token, head) row, the audio values ``av`` are
    N(0, 1); all rounded to bfloat16. Returns a dict with the fp32 values
    (``q, ak, av``), their bit patterns (``*_bits``) and ``face`` (int32).
    """
    La = w.audio_frames * w.audio_per_frame
    res = {}
    for name, shape, tid, norm in (
            ("q", (w.batch, w.n_tok, w.heads, w.head_dim), TENSOR_Q, True),
            ("ak", (w.batch, w.streams, La, w.heads, w.head_dim), TENSOR_K, True),
            ("av", (w.batch, w.streams, La, w.heads, w.head_dim), TENSOR_V, False)):
        vals, bits = draw_tensor(shape, wid=w.wid, b=0, chunk=w.first_frame, step=0, layer=layer,
                                 tensor_id=tid, rms_normalise=norm, dtype="bf16",
                                 base_seed=base_seed)
        res[name], res[name + "_bits"] = vals, bits
    res["face"] = face_ids(w.grid_h, w.grid_w, w.n_frames, w.streams, w.batch)
    return res


# --------------------------------------------------------------------------- rising scores


def draw_rising_sequence(wid: int, batch: int, n_tok: int, heads: int, head_dim: int, *,
                         cold_tokens: int, gamma_lo: float, gamma_hi: float, dtype: str,
                         base_seed: int = 0):
    """q, k, v ``[B, n_tok, H, D]`` whose scores rise steeply along the key
    positions: every query row is the RMS-normalised ``2 u + r`` for one random
    unit-RMS direction ``u`` per (batch, head) and noise ``r``; the keys at
    positions ``>= cold_tokens`` are ``gamma(p) u + r / 2`` with ``gamma``
    growing linearly from ``gamma_lo`` to ``gamma_hi`` over those positions,
    the first ``cold_tokens`` keys are RMS-normalised noise, values are N(0, 1).
    With the default scale a key at position p then scores about
    ``0.9 sqrt(D) gamma(p)`` against every query (log-e units), far above the
    first keys' scores. Returns the same dict as ``draw_qkv_sequence``.
    """
    res = {}
    per = {"q": [], "k": [], "v": []}
    for b in range(batch):
        rng = _rng(wid, b, FULL_SEQUENCE_CHUNK, 0, 0, 9, base_seed)
        u = rng.standard_normal((1, heads, head_dim), dtype=np.float32)
        u /= np.sqrt(np.mean(u * u, axis=-1, keepdims=True))
        q = 2.0 * u + rng.standard_normal((n_tok, heads, head_dim), dtype=np.float32)
        q /= np.sqrt(np.mean(q * q, axis=-1, keepdims=True))
        k = rng.standard_normal((n_tok, heads, head_dim), dtype=np.float32)
        k /= np.sqrt(np.mean(k * k, axis=-1, keepdims=True))
        hot = np.arange(n_tok) >= cold_tokens
        n_hot = int(hot.sum())
        if n_hot:
            gam = np.linspace(gamma_lo, gamma_hi, n_hot, dtype=np.float32)[:, None, None]
            k[hot] = gam * u + 0.5 * k[hot]
        v = rng.standard_normal((n_tok, heads, head_dim), dtype=np.float32)
        per["q"].append(q)
        per["k"].append(k)
        per["v"].append(v)
    for name, xs in per.items():
        x = np.stack(xs).astype(np.float32)
        if dtype == "bf16":
            bits = f32_to_bf16_bits(x)
            res[name], res[name + "_bits"] = bf16_bits_to_f32(bits), bits
        elif dtype == "f32":
            res[name] = x
        else:
            raise ValueError(f"unknown dtype {dtype!r}")
    return res
