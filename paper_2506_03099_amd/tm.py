"""ctypes binding of ``libtm.so`` (the C ABI in ``include/tm.h``).

Argument marshalling only: torch tensors supply device pointers, the current
HIP stream supplies the stream, and every step of the computation runs in the
library's HIP kernels. The binding raises if the library has not been built;
there is no other implementation to fall back to.

Function names match the C entry points.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtm.so")

TM_OK = 0
TM_E_ARG = -1
TM_E_SHAPE = -2
TM_E_DTYPE = -3
TM_E_ORDER = -4
TM_E_CAPACITY = -5
TM_E_DEVICE = -6
TM_F32 = 0
TM_BF16 = 1
TM_MAX_WINDOW = 12
TM_MAX_AUDIO_STREAMS = 32

STATUS_NAMES = {0: "TM_OK", -1: "TM_E_ARG", -2: "TM_E_SHAPE", -3: "TM_E_DTYPE",
                -4: "TM_E_ORDER", -5: "TM_E_CAPACITY", -6: "TM_E_DEVICE"}

_TORCH_DTYPE = {TM_F32: torch.float32, TM_BF16: torch.bfloat16}


class tm_attn_desc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("tokens_per_frame", ctypes.c_int32),
        ("chunk_frames", ctypes.c_int32),
        ("ref_frames", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
    ]

    @property
    def torch_dtype(self):
        return _TORCH_DTYPE[self.dtype]


class tm_audio_desc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("tokens_per_frame", ctypes.c_int32),
        ("audio_per_frame", ctypes.c_int32),
        ("audio_frames", ctypes.c_int32),
        ("streams", ctypes.c_int32),
        ("half_window", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
    ]


class TMError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load ``libtm.so`` (built by ``paper_2506_03099_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2506_03099_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        D = ctypes.POINTER(tm_attn_desc)
        AD = ctypes.POINTER(tm_audio_desc)
        sig = {
            "tm_kv_cache_tokens": (ctypes.c_int64, [D]),
            "tm_kv_cache_bytes": (ctypes.c_size_t, [D]),
            "tm_kv_cache_create": (ctypes.c_int, [D, P, P, ctypes.POINTER(P)]),
            "tm_kv_cache_destroy": (None, [P]),
            "tm_kv_cache_reset": (ctypes.c_int, [P]),
            "tm_kv_cache_locate": (ctypes.c_int, [P, ctypes.c_int32,
                                                  ctypes.POINTER(ctypes.c_int32),
                                                  ctypes.POINTER(ctypes.c_int32)]),
            "tm_kv_cache_latest": (ctypes.c_int32, [P]),
            "tm_kv_append": (ctypes.c_int, [P, ctypes.c_int32, P, P, ctypes.c_int32, P]),
            "tm_qkv_produce": (ctypes.c_int, [P, ctypes.c_int32, P, P, P, P, P, ctypes.c_float,
                                              P, ctypes.c_int32, P]),
            "tm_sparse_causal_attn_fwd": (ctypes.c_int, [D, P, ctypes.c_int32, P, P, P,
                                                         ctypes.c_int32, P, P, P]),
            "tm_sparse_causal_attn_fwd_f32out": (ctypes.c_int, [D, P, ctypes.c_int32, P, P, P,
                                                                ctypes.c_int32, P, P, P]),
            "tm_allowed_pairs": (ctypes.c_int64, [D, ctypes.c_int32, P, ctypes.c_int32]),
            "tm_audio_cross_attn_fwd": (ctypes.c_int, [AD, P, ctypes.c_int32, ctypes.c_int32, P, P,
                                                       P, P, P]),
            "tm_audio_cross_attn_fwd_f32out": (ctypes.c_int, [AD, P, ctypes.c_int32,
                                                              ctypes.c_int32, P, P, P, P, P]),
            "tm_sparse_causal_attn_bwd": (ctypes.c_int, [D, ctypes.c_int32, P, P, P, P, P, P, P,
                                                         P, P, P, P]),
            "tm_sparse_causal_attn_bwd_noalloc": (ctypes.c_int, [D, ctypes.c_int32, P, P, P, P, P,
                                                                 P, P, P, P, P]),
            "tm_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def tm_last_error() -> str:
    return lib().tm_last_error().decode()


def _check(status: int):
    if status != TM_OK:
        raise TMError(status, tm_last_error())


def make_desc(batch, heads, head_dim, tokens_per_frame, chunk_frames, ref_frames, window,
              dtype, softmax_scale=0.0) -> tm_attn_desc:
    if isinstance(dtype, torch.dtype):
        dtype = {torch.float32: TM_F32, torch.bfloat16: TM_BF16}[dtype]
    elif isinstance(dtype, str):
        dtype = {"f32": TM_F32, "bf16": TM_BF16}[dtype]
    return tm_attn_desc(batch, heads, head_dim, tokens_per_frame, chunk_frames, ref_frames,
                        window, dtype, softmax_scale)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise TMError(TM_E_ARG, "tensor is not on a GPU")
    if not t.is_contiguous():
        raise TMError(TM_E_ARG, "tensor is not contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def tm_kv_cache_tokens(desc: tm_attn_desc) -> int:
    return lib().tm_kv_cache_tokens(ctypes.byref(desc))


def tm_kv_cache_bytes(desc: tm_attn_desc) -> int:
    return lib().tm_kv_cache_bytes(ctypes.byref(desc))


def tm_allowed_pairs(desc: tm_attn_desc, q_chunk: int, cache=None, n_frames: int = 0) -> int:
    h = cache.handle if cache is not None else None
    return lib().tm_allowed_pairs(ctypes.byref(desc), q_chunk, h, n_frames)


class KVCache:
    """A ``tm_kv_cache`` handle together with the torch tensors that own its
    pools: K ``[B, H, capacity, D]``, V ``[B, H, capacity // 64, D, 64]``
    (64-token blocks stored dimension-major)."""

    def __init__(self, desc: tm_attn_desc, device="cuda", k_pool=None, v_pool=None):
        self.desc = desc
        cap = tm_kv_cache_tokens(desc)
        if cap <= 0:
            raise TMError(TM_E_SHAPE, "invalid descriptor")
        B, H, D, dt = desc.batch, desc.heads, desc.head_dim, desc.torch_dtype
        self.k_pool = k_pool if k_pool is not None else torch.empty(
            (B, H, cap, D), dtype=dt, device=device)
        self.v_pool = v_pool if v_pool is not None else torch.empty(
            (B, H, cap // 64, D, 64), dtype=dt, device=device)
        h = ctypes.c_void_p()
        _check(lib().tm_kv_cache_create(ctypes.byref(desc), _ptr(self.k_pool), _ptr(self.v_pool),
                                        ctypes.byref(h)))
        self.handle = h

    @property
    def capacity(self) -> int:
        return self.k_pool.shape[2]

    def close(self):
        if getattr(self, "handle", None) is not None and _lib is not None:
            _lib.tm_kv_cache_destroy(self.handle)
            self.handle = None

    __del__ = close

    def latest(self) -> int:
        return lib().tm_kv_cache_latest(self.handle)

    def locate(self, chunk: int):
        off, n = ctypes.c_int32(), ctypes.c_int32()
        _check(lib().tm_kv_cache_locate(self.handle, chunk, ctypes.byref(off), ctypes.byref(n)))
        return off.value, n.value

    def reset(self):
        _check(lib().tm_kv_cache_reset(self.handle))


def tm_kv_cache_create(desc: tm_attn_desc, device="cuda", k_pool=None, v_pool=None) -> KVCache:
    return KVCache(desc, device, k_pool, v_pool)


def tm_kv_append(cache: KVCache, chunk: int, k, v, n_tok: int | None = None, stream=None):
    """Append chunk ``chunk``'s K/V (``[B, n_tok, H, D]``) to the cache."""
    if n_tok is None:
        n_tok = k.shape[1]
    _check(lib().tm_kv_append(cache.handle, chunk, _ptr(k), _ptr(v), n_tok, _stream(stream)))


def tm_qkv_produce(cache: KVCache, chunk: int, q, k, v, q_gain=None, k_gain=None,
                   eps: float = 0.0, q_out=None, n_tok: int | None = None, stream=None):
    """RMS-normalise the chunk's q and k rows and append k (normalised) and v
    to the cache; returns ``q_out`` (allocated like q if not given)."""
    if n_tok is None:
        n_tok = k.shape[1]
    if q_out is None:
        q_out = torch.empty_like(q)
    _check(lib().tm_qkv_produce(cache.handle, chunk, _ptr(q), _ptr(k), _ptr(v), _ptr(q_gain),
                                _ptr(k_gain), eps, _ptr(q_out), n_tok, _stream(stream)))
    return q_out


def tm_sparse_causal_attn_fwd(desc: tm_attn_desc, q, q_chunk: int, cache: KVCache | None = None,
                              k=None, v=None, n_frames: int = 0, o=None, lse=None,
                              stream=None):
    """Sparse causal attention; returns ``o`` (allocated like q if not given)."""
    if o is None:
        o = torch.empty_like(q)
    h = cache.handle if cache is not None else None
    _check(lib().tm_sparse_causal_attn_fwd(ctypes.byref(desc), _ptr(q), q_chunk, h, _ptr(k),
                                           _ptr(v), n_frames, _ptr(o), _ptr(lse),
                                           _stream(stream)))
    return o


def tm_sparse_causal_attn_fwd_f32out(desc: tm_attn_desc, q, q_chunk: int,
                                     cache: KVCache | None = None, k=None, v=None,
                                     n_frames: int = 0, o=None, lse=None, stream=None):
    """The same attention with an fp32 output (``o`` allocated as fp32 like q
    if not given); returns ``o``."""
    if o is None:
        o = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    h = cache.handle if cache is not None else None
    _check(lib().tm_sparse_causal_attn_fwd_f32out(ctypes.byref(desc), _ptr(q), q_chunk, h, _ptr(k),
                                                  _ptr(v), n_frames, _ptr(o), _ptr(lse),
                                                  _stream(stream)))
    return o


def make_audio_desc(batch, heads, head_dim, tokens_per_frame, audio_per_frame, audio_frames,
                    streams=1, half_window=2, dtype="bf16", softmax_scale=0.0) -> tm_audio_desc:
    if isinstance(dtype, torch.dtype):
        dtype = {torch.float32: TM_F32, torch.bfloat16: TM_BF16}[dtype]
    elif isinstance(dtype, str):
        dtype = {"f32": TM_F32, "bf16": TM_BF16}[dtype]
    return tm_audio_desc(batch, heads, head_dim, tokens_per_frame, audio_per_frame, audio_frames,
                         streams, half_window, dtype, softmax_scale)


def tm_audio_cross_attn_fwd(desc: tm_audio_desc, q, first_frame: int, ak, av, face, o=None,
                            n_tok: int | None = None, stream=None):
    """Audio cross-attention of the query rows ``q`` ([B, n_tok, H, D], row i
    in latent frame first_frame + i // T) over the audio keys/values ``ak``,
    ``av`` ([B, M, F_a * A, H, D]) with int32 face ids ``face`` ([B, n_tok]);
    returns ``o`` (allocated like q if not given)."""
    if n_tok is None:
        n_tok = q.shape[1]
    if o is None:
        o = torch.empty_like(q)
    _check(lib().tm_audio_cross_attn_fwd(ctypes.byref(desc), _ptr(q), first_frame, n_tok, _ptr(ak),
                                         _ptr(av), _ptr(face), _ptr(o), _stream(stream)))
    return o


def tm_audio_cross_attn_fwd_f32out(desc: tm_audio_desc, q, first_frame: int, ak, av, face,
                                   o=None, n_tok: int | None = None, stream=None):
    """The audio cross-attention with an fp32 output; returns ``o``."""
    if n_tok is None:
        n_tok = q.shape[1]
    if o is None:
        o = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check(lib().tm_audio_cross_attn_fwd_f32out(ctypes.byref(desc), _ptr(q), first_frame, n_tok,
                                                _ptr(ak), _ptr(av), _ptr(face), _ptr(o),
                                                _stream(stream)))
    return o


def tm_sparse_causal_attn_bwd(desc: tm_attn_desc, n_frames: int, q, k, v, o, lse, dout, delta=None,
                              dq=None, dk=None, dv=None, stream=None):
    """Gradients (dq, dk, dv) of the full-sequence sparse causal attention;
    ``delta`` is an fp32 [B, H, L] workspace (allocated if not given)."""
    if delta is None:
        delta = torch.empty_like(lse)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _check(lib().tm_sparse_causal_attn_bwd(ctypes.byref(desc), n_frames, _ptr(q), _ptr(k), _ptr(v),
                                           _ptr(o), _ptr(lse), _ptr(dout), _ptr(delta), _ptr(dq),
                                           _ptr(dk), _ptr(dv), _stream(stream)))
    return dq, dk, dv


def tm_sparse_causal_attn_bwd_noalloc(desc: tm_attn_desc, n_frames: int, q, k, v, o, lse, dout,
                                      dq, dk, dv, stream=None):
    """The backward with the library's device-global workspace: the caller
    passes every output (nothing is allocated); returns (dq, dk, dv)."""
    _check(lib().tm_sparse_causal_attn_bwd_noalloc(ctypes.byref(desc), n_frames, _ptr(q), _ptr(k),
                                                   _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
                                                   _ptr(dq), _ptr(dk), _ptr(dv), _stream(stream)))
    return dq, dk, dv
