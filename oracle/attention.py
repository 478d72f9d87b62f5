"""Dense masked attention: the oracle for the sparse causal attention
(test infrastructure only; never imported by the product path).

Paper: TalkingMachines, Sec. 4.2, the attention equation
    Attention(Q_t, K, V) = softmax(Q_t K^T / sqrt(d)) V,
with K and V holding only the tokens of {c_0, c_{t-1}, c_t}. The method is
exact attention over that key set, so the oracle is the definition written out:
materialise every logit, set the disallowed ones to -inf through an explicit
boolean mask, take a row softmax, zero the disallowed probabilities, multiply
by V. No tiling, no online softmax, no reordering.

Readings: d is the head dimension (scale 1/sqrt(head_dim) unless given);
arithmetic is fp32 (the precision the method is stated against) unless the
caller asks for fp64; inputs are exactly the values the device sees (bf16
inputs arrive here already widened to fp32 without rounding).
"""
from __future__ import annotations

import numpy as np

from .geometry import ChunkGeometry, allowed_mask


def masked_attention(q, k, v, mask, scale, *, dtype=np.float32, return_probs=False):
    """Attention of one head.

    q: [Lq, D], k and v: [Lk, D], mask: [Lq, Lk] bool (True = may attend).
    Returns (o [Lq, D], lse [Lq]) where lse is the natural-log normaliser
    log(sum_j exp(scale * q_i . k_j)) over the allowed keys; with
    ``return_probs`` also the probability matrix P [Lq, Lk].
    Every row must allow at least one key.
    """
    q = np.asarray(q, dtype=dtype)
    k = np.asarray(k, dtype=dtype)
    v = np.asarray(v, dtype=dtype)
    s = (q @ k.T) * dtype(scale)
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    if not np.all(np.isfinite(m)):
        raise ValueError("a query row has no allowed key")
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    p = e / z
    p = np.where(mask, p, dtype(0))
    o = p @ v
    lse = m[:, 0] + np.log(z[:, 0])
    if return_probs:
        return o, lse, p
    return o, lse


def _default_scale(head_dim: int) -> float:
    return 1.0 / float(np.sqrt(head_dim))


def full_sequence_attention(q, k, v, g: ChunkGeometry, *, scale=None, q_offset: int = 0,
                            heads=None, rows=None, row_block: int = 2048,
                            dtype=np.float32):
    """Sparse causal attention of a whole latent sequence (full-sequence form).

    q: [B, Lq, H, D] whose row i sits at position ``q_offset + i``;
    k, v: [B, Lk, H, D] at positions 0 .. Lk-1.
    ``heads`` / ``rows`` optionally select a subset of heads / query rows (for
    sampled comparisons at large sizes). Rows are processed in blocks of
    ``row_block``; each row is still a complete masked row.
    Returns (o [B, n_rows, n_heads, D], lse [B, n_heads, n_rows]).
    """
    B, Lq, H, D = q.shape
    Lk = k.shape[1]
    if scale is None:
        scale = _default_scale(D)
    heads = list(range(H)) if heads is None else list(heads)
    rows = np.arange(Lq) if rows is None else np.asarray(rows, dtype=np.int64)
    k_pos = np.arange(Lk)
    o = np.empty((B, len(rows), len(heads), D), dtype=dtype)
    lse = np.empty((B, len(heads), len(rows)), dtype=dtype)
    for b in range(B):
        for hi, h in enumerate(heads):
            kh = np.ascontiguousarray(k[b, :, h, :])
            vh = np.ascontiguousarray(v[b, :, h, :])
            for r0 in range(0, len(rows), row_block):
                sel = rows[r0:r0 + row_block]
                mask = allowed_mask(q_offset + sel, k_pos, g)
                ob, lb = masked_attention(q[b, sel, h, :], kh, vh, mask, scale, dtype=dtype)
                o[b, r0:r0 + len(sel), hi, :] = ob
                lse[b, hi, r0:r0 + len(sel)] = lb
    return o, lse


def chunk_start(chunk: int, g: ChunkGeometry) -> int:
    """Position of the first token of chunk ``chunk`` in the latent sequence."""
    if chunk == 0:
        return 0
    return g.ref_frames * g.tokens_per_frame + (chunk - 1) * g.chunk_frames * g.tokens_per_frame


class StreamHistory:
    """Streaming form: the K/V of every chunk appended so far, kept whole.

    Paper: Sec. 4.3, "KV & Embedding Cachings": at inference the K/V of c_0 and
    c_{t-1} are cached for each timestep and every transformer block, so the
    context is never recomputed. This oracle does not model a cache at all: it
    keeps the complete history of appended chunks at their sequence positions
    and lets the mask pick the keys, so a device cache that evicts the wrong
    chunk, or keeps one it should have dropped, disagrees with it.

    Append rules: the reference chunk 0 comes first; after that a chunk index
    equal to the latest one replaces it (the step-2 overwrite of a shared
    cache) and latest + 1 advances the stream.

    One history is one (denoising step, layer) instance. That the paper keeps a
    separate cache per timestep, filled while the context chunk was itself
    being denoised at that timestep, is a reading of "for each timestep" that no
    number in the paper checks: parity unpinned for that reading (the
    attention arithmetic itself is pinned).
    """

    def __init__(self, g: ChunkGeometry):
        self.g = g
        self.k: dict[int, np.ndarray] = {}
        self.v: dict[int, np.ndarray] = {}
        self.latest = -1

    def append(self, chunk: int, k, v):
        """k, v: [B, n_tok, H, D] for chunk ``chunk``."""
        if self.latest < 0:
            if chunk != 0:
                raise ValueError("the reference chunk 0 must be appended first")
        elif chunk not in (self.latest, self.latest + 1):
            raise ValueError(f"chunk {chunk} after {self.latest}")
        self.k[chunk] = np.array(k, copy=True)
        self.v[chunk] = np.array(v, copy=True)
        self.latest = chunk

    def keys(self):
        """All appended K/V concatenated with their positions."""
        order = sorted(self.k)
        pos = np.concatenate([chunk_start(c, self.g) + np.arange(self.k[c].shape[1])
                              for c in order])
        k = np.concatenate([self.k[c] for c in order], axis=1)
        v = np.concatenate([self.v[c] for c in order], axis=1)
        return pos, k, v

    def attend(self, q, q_chunk: int, *, scale=None, heads=None, rows=None,
               dtype=np.float32):
        """Attention of chunk ``q_chunk``'s queries q [B, n, H, D] over the history.

        Returns (o [B, n_rows, n_heads, D], lse [B, n_heads, n_rows]).
        """
        B, n, H, D = q.shape
        if scale is None:
            scale = _default_scale(D)
        heads = list(range(H)) if heads is None else list(heads)
        rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
        k_pos, k, v = self.keys()
        q_pos = chunk_start(q_chunk, self.g) + rows
        mask = allowed_mask(q_pos, k_pos, self.g)
        o = np.empty((B, len(rows), len(heads), D), dtype=dtype)
        lse = np.empty((B, len(heads), len(rows)), dtype=dtype)
        for b in range(B):
            for hi, h in enumerate(heads):
                ob, lb = masked_attention(q[b, rows, h, :], k[b, :, h, :], v[b, :, h, :],
                                          mask, scale, dtype=dtype)
                o[b, :, hi, :] = ob
                lse[b, hi, :] = lb
        return o, lse
