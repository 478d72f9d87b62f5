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


def sampled_sequence_attention_backward(q, k, v, do, g: ChunkGeometry, *, q_rows, k_rows,
                                        heads=None, scale=None, row_block: int = 1024,
                                        dtype=np.float64):
    """Selected gradient rows of the whole-sequence backward, for sequences
    whose L x L matrices do not fit in memory.

    The same chain rule as ``masked_attention_backward``, evaluated in blocks
    of ``row_block`` query rows; every query row is always a complete masked
    row over all L keys. Two passes per (batch, head):

    1. for every query row i: P_i (masked row softmax of scale q_i K^T),
       dP_i = dO_i V^T and g_i = sum_j P_ij dP_ij, kept as lse_i =
       log sum_j exp(scale q_i.k_j) and g_i;
    2. dQ_i = scale dS_i K for i in ``q_rows``, with dS_i = P_i * (dP_i - g_i);
       dK_j = scale sum_i dS_ij q_i and dV_j = sum_i P_ij dO_i for j in
       ``k_rows``, summing over every query row (P_ij = exp(s_ij - lse_i),
       the row softmax written with its normaliser).

    Returns ((dq, dk, dv), (mq, mk, mv)): dq and mq [B, len(q_rows), n_heads,
    D], the others [B, len(k_rows), n_heads, D]; the m's are the sums of
    absolute products as in ``masked_attention_backward``.
    """
    B, L, H, D = q.shape
    if scale is None:
        scale = 1.0 / float(np.sqrt(D))
    sc = dtype(scale)
    heads = list(range(H)) if heads is None else list(heads)
    q_rows = np.asarray(q_rows, dtype=np.int64)
    k_rows = np.asarray(k_rows, dtype=np.int64)
    pos = np.arange(L)
    nh = len(heads)
    dq = np.zeros((B, len(q_rows), nh, D), dtype=dtype)
    mq = np.zeros_like(dq)
    dk = np.zeros((B, len(k_rows), nh, D), dtype=dtype)
    mk, dv, mv = np.zeros_like(dk), np.zeros_like(dk), np.zeros_like(dk)
    for b in range(B):
        for hi, h in enumerate(heads):
            qh, kh, vh, doh = (np.ascontiguousarray(x[b, :, h, :], dtype=dtype) for x in (q, k, v, do))
            lse = np.empty(L, dtype=dtype)
            gsum = np.empty(L, dtype=dtype)
            for r0 in range(0, L, row_block):
                rows = pos[r0:r0 + row_block]
                mask = allowed_mask(rows, pos, g)
                s = np.where(mask, (qh[rows] @ kh.T) * sc, -np.inf)
                m = s.max(axis=1, keepdims=True)
                e = np.where(mask, np.exp(s - m), dtype(0))
                z = e.sum(axis=1, keepdims=True)
                p = e / z
                dp = doh[rows] @ vh.T
                lse[rows] = m[:, 0] + np.log(z[:, 0])
                gsum[rows] = (p * dp).sum(axis=1)
            # dQ of the selected query rows
            mask = allowed_mask(q_rows, pos, g)
            s = np.where(mask, (qh[q_rows] @ kh.T) * sc, -np.inf)
            p = np.where(mask, np.exp(s - lse[q_rows, None]), dtype(0))
            ds = p * (doh[q_rows] @ vh.T - gsum[q_rows, None])
            dq[b, :, hi] = sc * (ds @ kh)
            mq[b, :, hi] = sc * (np.abs(ds) @ np.abs(kh))
            # dK, dV of the selected keys, summed over every query row
            ks, vs = kh[k_rows], vh[k_rows]
            for r0 in range(0, L, row_block):
                rows = pos[r0:r0 + row_block]
                mask = allowed_mask(rows, k_rows, g)
                s = np.where(mask, (qh[rows] @ ks.T) * sc, -np.inf)
                p = np.where(mask, np.exp(s - lse[rows, None]), dtype(0))
                ds = p * (doh[rows] @ vs.T - gsum[rows, None])
                dk[b, :, hi] += sc * (ds.T @ qh[rows])
                mk[b, :, hi] += sc * (np.abs(ds).T @ np.abs(qh[rows]))
                dv[b, :, hi] += p.T @ doh[rows]
                mv[b, :, hi] += p.T @ np.abs(doh[rows])
    return (dq, dk, dv), (mq, mk, mv)
