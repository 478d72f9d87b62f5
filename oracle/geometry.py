"""Chunk geometry and the sparse causal key set (oracle; test infrastructure only).

Paper: TalkingMachines, Sec. 4.2. The latent sequence of a clip (21 latent
frames for 81 video frames) is divided into chunks of 3 latent frames
("Chunked Processing"); a token of chunk c_t attends to every token of c_t,
of the previous chunk c_{t-1} and of the starting chunk c_0, which holds the
ground-truth image ("Sparse Attention Pattern"); attention inside a chunk is
bidirectional and across chunks causal (first paragraph of Sec. 4.2).

Readings taken where the paper leaves a choice open:

* c_0 is the first ``R`` latent frames (the reference frames); the chunk
  length ``C`` applies to the frames after it. The workloads use R = 1 (the
  image frame) and C = 3; R = C = 3 gives the literal "7 chunks of 3".
* A final chunk shorter than C frames sits at the end of the sequence.
* The window of previous chunks is a parameter ``W`` (the paper: W = 1).
  For t = 1 the previous chunk is c_0 itself; the key set is a set, so no key
  is counted twice.
* Queries of c_0 see c_0 only (the rule with t = 0).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ChunkGeometry:
    tokens_per_frame: int  # T: latent tokens per latent frame
    chunk_frames: int  # C: latent frames per chunk after c_0
    ref_frames: int  # R: latent frames in the starting chunk c_0
    window: int = 1  # W: previous chunks a chunk may see besides c_0

    def __post_init__(self):
        if min(self.tokens_per_frame, self.chunk_frames, self.ref_frames) < 1:
            raise ValueError("T, C and R must be >= 1")
        if self.window < 0:
            raise ValueError("W must be >= 0")


def chunk_of_frame(frame, g: ChunkGeometry):
    """Chunk index of latent frame(s) ``frame``: 0 for the reference frames,
    then 1, 2, ... for consecutive groups of C frames."""
    f = np.asarray(frame, dtype=np.int64)
    return np.where(f < g.ref_frames, 0, 1 + (f - g.ref_frames) // g.chunk_frames)


def chunk_of_position(pos, g: ChunkGeometry):
    """Chunk index of token position(s) ``pos`` in the latent sequence."""
    return chunk_of_frame(np.asarray(pos, dtype=np.int64) // g.tokens_per_frame, g)


def allowed_mask(q_pos, k_pos, g: ChunkGeometry) -> np.ndarray:
    """Explicit boolean mask M[i, j]: may the query at position q_pos[i] see
    the key at position k_pos[j]?

    True iff the key's chunk is c_0, or lies between the query's own chunk a
    and a - W (inclusive), i.e. {c_0, c_{a-W}, ..., c_{a-1}, c_a}.
    """
    a = chunk_of_position(q_pos, g)[:, None]
    c = chunk_of_position(k_pos, g)[None, :]
    return (c == 0) | ((c >= a - g.window) & (c <= a))


def allowed_pair_count(n_tokens: int, g: ChunkGeometry) -> int:
    """Number of allowed (query, key) pairs when a sequence of ``n_tokens``
    attends to itself (the count the FLOP figures are based on)."""
    pos = np.arange(n_tokens)
    total = 0
    for i0 in range(0, n_tokens, 4096):
        total += int(allowed_mask(pos[i0:i0 + 4096], pos, g).sum())
    return total
