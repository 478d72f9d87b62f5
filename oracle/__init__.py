"""Plain CPU oracle for the sparse causal attention of the chunked autoregressive
student in TalkingMachines (arXiv 2506.03099).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or link
this package: only the test suite, the smoke check and the benchmark's CPU
baseline leg use it. It shares no code with the GPU path (no kernels, headers,
helpers or constant tables); the only code both sides use is the seeded input
generator in ``synth``.

What it computes, and where the paper defines it:

* ``geometry``  -- latent frames grouped into chunks, the starting chunk c_0
  holding the reference image, and which keys a query may see: its own chunk
  c_t (bidirectionally), the previous chunk c_{t-1} and c_0 (Sec. 4.2,
  "Chunked Processing" and "Sparse Attention Pattern"; the same rule restated
  among the DMD modifications as "Sparse Causal Attention").
* ``attention`` -- exact attention softmax(Q_t K^T / sqrt(d)) V with K and V
  restricted to {c_0, c_{t-1}, c_t} (Sec. 4.2, the attention equation), as a
  dense fp32 computation over an explicit boolean mask, in the full-sequence
  form and in the streaming form that keeps every appended chunk's K/V on the
  host (Sec. 4.3, "KV & Embedding Cachings").
* ``brute``     -- an independent fp64 per-query enumeration of the same key
  set, used to pin ``attention`` on tiny inputs, and an fp64 per-element
  loop of the gradients and of their absolute-product sums, used to pin
  ``backward``.
* ``producer``  -- the RMS normalisation of query and key rows that precedes
  the attention and the KV cache (the fused K/V producer).
* ``backward``  -- the gradients dQ, dK, dV of the sparse causal attention
  (for training the student through it), from the chain rule over the
  masked row softmax.
* ``audio``     -- the audio cross-attention of Sec. 4.1: each latent frame's
  tokens attend to the audio tokens of the five frames centred on it, face
  tokens only, each face to its own audio stream.

Every function here is pinned by the ``-m "not gpu"`` tests against closed
forms, invariants, library special cases and the brute force; the one reading
no number in the paper can check (one cache per denoising step) is marked
"parity unpinned" in ``attention``.
"""
from .geometry import (  # noqa: F401
    ChunkGeometry,
    chunk_of_frame,
    chunk_of_position,
    allowed_mask,
    allowed_pair_count,
)
from .attention import (  # noqa: F401
    masked_attention,
    full_sequence_attention,
    StreamHistory,
)
from .brute import brute_force_attention, brute_force_backward  # noqa: F401
from .producer import rms_normalise  # noqa: F401
from .audio import audio_cross_attention, audio_window  # noqa: F401
from .backward import (  # noqa: F401
    masked_attention_backward,
    full_sequence_attention_backward,
    sampled_sequence_attention_backward,
)
