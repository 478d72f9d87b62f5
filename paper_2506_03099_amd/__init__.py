"""Sparse causal streaming attention for MI355X (gfx950).

The computation that dominates inference in the chunked autoregressive
video-diffusion student of TalkingMachines (arXiv 2506.03099): block-sparse
causal attention over {c_0, c_{t-1}, c_t} and the KV-cache append that lets the
denoising steps reuse cached context, as hand-written HIP kernels behind the C
ABI of ``include/tm.h``. ``tm`` is the ctypes binding.
"""
from . import tm  # noqa: F401
from .tm import (  # noqa: F401
    KVCache,
    TMError,
    make_desc,
    tm_allowed_pairs,
    tm_kv_append,
    tm_kv_cache_bytes,
    tm_kv_cache_create,
    tm_kv_cache_tokens,
    tm_last_error,
    tm_sparse_causal_attn_fwd,
)
