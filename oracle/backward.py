"""Oracle of the backward pass of the sparse causal attention (test
infrastructure only; never imported by the product path).

Paper: TalkingMachines, Sec. 4.2. The student is trained (the DMD stage
with "Sparse Causal Attention") through the attention of Sec. 4.2,
O = softmax(scale * Q K^T) V over each query's allowed key set
{c_0, c_{a-W}, ..., c_a}. Training needs the gradients of a loss L with
respect to Q, K and V given dO = dL/dO. They follow from the chain rule,
written out here for one head, with P the masked row softmax:

    dV = P^T dO
    dP = dO V^T
    dS = P * (dP - rowsum(P * dP))          (softmax Jacobian, row by row)
    dQ = scale * dS K
    dK = scale * dS^T Q

rowsum(P * dP) equals rowsum(dO * O) because O = P V. Disallowed pairs have
P = 0 and so dS = 0: no gradient flows through them. Computed in float64 over
an explicit boolean mask, materialising every matrix; no tiling.
"""
from __future__ import annotations

import numpy as np

from .geometry import ChunkGeometry, allowed_mask


def masked_attention_backward(q, k, v, do, mask, scale, *, dtype=np.float64, magnitudes=False):
    """Gradients of one head.

    q, do: [Lq, D]; k, v: [Lk, D]; mask: [Lq, Lk] bool (True = may attend).
    Returns (dq [Lq, D], dk [Lk, D], dv [Lk, D]). Every row must allow a key.
    With ``magnitudes`` also the sums of absolute products behind each
    gradient element, scale |dS| |K|, scale |dS|^T |Q| and |P|^T |dO|: a sum
    whose factors each carry a relative error e has an error of at most e
    times that sum.
    """
    q, k, v, do = (np.asarray(x, dtype=dtype) for x in (q, k, v, do))
    s = (q @ k.T) * dtype(scale)
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    if not np.all(np.isfinite(m)):
        raise ValueError("a query row has no allowed key")
    e = np.where(mask, np.exp(s - m), dtype(0))
    p = e / e.sum(axis=1, keepdims=True)
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    dq = dtype(scale) * (ds @ k)
    dk = dtype(scale) * (ds.T @ q)
    if magnitudes:
        a = np.abs(ds)
        return (dq, dk, dv), (dtype(scale) * (a @ np.abs(k)), dtype(scale) * (a.T @ np.abs(q)),
                              p.T @ np.abs(do))
    return dq, dk, dv


def full_sequence_attention_backward(q, k, v, do, g: ChunkGeometry, *, scale=None, heads=None,
                                     dtype=np.float64, magnitudes=False):
    """Gradients of the sparse causal attention of a whole latent sequence.

    q, k, v, do: [B, L, H, D] (position i = token i). ``heads`` optionally
    selects a subset. Returns (dq, dk, dv), each [B, L, n_heads, D]; with
    ``magnitudes`` also the three absolute-product sums, same shapes.
    """
    B, L, H, D = q.shape
    if scale is None:
        scale = 1.0 / float(np.sqrt(D))
    heads = list(range(H)) if heads is None else list(heads)
    pos = np.arange(L)
    mask = allowed_mask(pos, pos, g)
    n_out = 6 if magnitudes else 3
    out = [np.empty((B, L, len(heads), D), dtype=dtype) for _ in range(n_out)]
    for b in range(B):
        for hi, h in enumerate(heads):
            res = masked_attention_backward(q[b, :, h], k[b, :, h], v[b, :, h], do[b, :, h],
                                            mask, scale, dtype=dtype, magnitudes=magnitudes)
            grads = res[0] + res[1] if magnitudes else res
            for o, gr in zip(out, grads):
                o[b, :, hi] = gr
    if magnitudes:
        return tuple(out[:3]), tuple(out[3:])
    return tuple(out)
