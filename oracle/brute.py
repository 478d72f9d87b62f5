"""Brute-force fp64 sparse causal attention, one query at a time (oracle;
test infrastructure only).

Built independently of ``geometry`` and ``attention`` so that each pins the
other on tiny inputs: the chunks are laid out as explicit lists of token
positions, the key set of a query is the union of the token lists of
{c_0} and {c_{a-W}, ..., c_a} as a Python set (TalkingMachines, Sec. 4.2,
"Sparse Attention Pattern"; the set semantics make c_{t-1} = c_0 at t = 1 count
once), and the softmax is evaluated in fp64 with ``math.exp`` and
``math.fsum`` (Sec. 4.2, the attention equation).
"""
from __future__ import annotations

import math

import numpy as np


def chunk_token_lists(n_tokens: int, T: int, C: int, R: int):
    """Token positions of each chunk: c_0 = the first R frames, then groups of
    C frames, the last group possibly shorter."""
    chunks = [list(range(0, min(R * T, n_tokens)))]
    start = R * T
    while start < n_tokens:
        chunks.append(list(range(start, min(start + C * T, n_tokens))))
        start += C * T
    return chunks


def brute_force_attention(q, k, v, *, T: int, C: int, R: int, W: int, scale=None,
                          q_positions=None, k_positions=None):
    """q: [Lq, D]; k, v: [Lk, D] (one head). Positions default to 0..L-1.

    Returns (o [Lq, D] fp64, lse [Lq] fp64, key_sets list of sorted key index
    lists).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, D = q.shape
    Lk = k.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    q_positions = list(range(Lq)) if q_positions is None else [int(p) for p in q_positions]
    k_positions = list(range(Lk)) if k_positions is None else [int(p) for p in k_positions]
    n_tokens = max(max(q_positions), max(k_positions)) + 1
    chunks = chunk_token_lists(n_tokens, T, C, R)
    chunk_of = {}
    for ci, toks in enumerate(chunks):
        for p in toks:
            chunk_of[p] = ci
    index_of_key_pos = {}
    for j, p in enumerate(k_positions):
        index_of_key_pos.setdefault(p, []).append(j)

    o = np.zeros((Lq, D))
    lse = np.zeros(Lq)
    key_sets = []
    for i, p in enumerate(q_positions):
        a = chunk_of[p]
        visible_chunks = {0} | set(range(max(0, a - W), a + 1))
        visible_pos = set()
        for ci in visible_chunks:
            visible_pos.update(chunks[ci])
        keys = sorted(j for pp in visible_pos for j in index_of_key_pos.get(pp, []))
        key_sets.append(keys)
        logits = [scale * math.fsum(q[i, d] * k[j, d] for d in range(D)) for j in keys]
        mx = max(logits)
        w = [math.exp(x - mx) for x in logits]
        z = math.fsum(w)
        for d in range(D):
            o[i, d] = math.fsum(w[n] * v[j, d] for n, j in enumerate(keys)) / z
        lse[i] = mx + math.log(z)
    return o, lse, key_sets


def brute_force_backward(q, k, v, do, *, T: int, C: int, R: int, W: int, scale=None):
    """Gradients of the loss sum(O * dO) of one head, one element at a time in
    fp64 (``math.exp``, ``math.fsum``), with the key sets enumerated as above.

    Written independently of ``backward``: for each query i with key set K_i,
        s_ij = scale q_i.k_j,  p_ij = exp(s_ij - max) / sum,
        dp_ij = dO_i.v_j,      g_i = sum_j p_ij dp_ij,
        ds_ij = p_ij (dp_ij - g_i)            (row Jacobian of the softmax),
    and the three gradients, each with the sum of the absolute values of the
    products it adds up (the bound on its rounding error when every factor
    carries a relative error):
        dQ_id = scale sum_j ds_ij k_jd        |  scale sum_j |ds_ij| |k_jd|
        dK_jd = scale sum_i ds_ij q_id        |  scale sum_i |ds_ij| |q_id|
        dV_jd = sum_i p_ij dO_id              |  sum_i p_ij |dO_id|
    (TalkingMachines, Sec. 4.2: the attention equation over {c_0, c_{a-W}, ..,
    c_a}, differentiated for training the student through it.)

    q, k, v, do: [L, D] at positions 0..L-1. Returns ((dq, dk, dv), (mq, mk, mv)),
    all [L, D] fp64.
    """
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    L, D = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    chunks = chunk_token_lists(L, T, C, R)
    chunk_of = {p: ci for ci, toks in enumerate(chunks) for p in toks}
    dq, mq = np.zeros((L, D)), np.zeros((L, D))
    dk_terms = [[[] for _ in range(D)] for _ in range(L)]
    mk_terms = [[[] for _ in range(D)] for _ in range(L)]
    dv_terms = [[[] for _ in range(D)] for _ in range(L)]
    mv_terms = [[[] for _ in range(D)] for _ in range(L)]
    for i in range(L):
        a = chunk_of[i]
        keys = set()
        for ci in {0} | set(range(max(0, a - W), a + 1)):
            keys.update(chunks[ci])
        keys = sorted(keys)
        logits = [scale * math.fsum(q[i, d] * k[j, d] for d in range(D)) for j in keys]
        mx = max(logits)
        w = [math.exp(x - mx) for x in logits]
        z = math.fsum(w)
        p = [x / z for x in w]
        dp = [math.fsum(do[i, d] * v[j, d] for d in range(D)) for j in keys]
        gi = math.fsum(pn * dpn for pn, dpn in zip(p, dp))
        ds = [pn * (dpn - gi) for pn, dpn in zip(p, dp)]
        for d in range(D):
            dq[i, d] = scale * math.fsum(ds[n] * k[j, d] for n, j in enumerate(keys))
            mq[i, d] = scale * math.fsum(abs(ds[n]) * abs(k[j, d]) for n, j in enumerate(keys))
        for n, j in enumerate(keys):
            for d in range(D):
                dk_terms[j][d].append(ds[n] * q[i, d])
                mk_terms[j][d].append(abs(ds[n]) * abs(q[i, d]))
                dv_terms[j][d].append(p[n] * do[i, d])
                mv_terms[j][d].append(p[n] * abs(do[i, d]))
    dk = np.array([[scale * math.fsum(t) for t in row] for row in dk_terms])
    mk = np.array([[scale * math.fsum(t) for t in row] for row in mk_terms])
    dv = np.array([[math.fsum(t) for t in row] for row in dv_terms])
    mv = np.array([[math.fsum(t) for t in row] for row in mv_terms])
    return (dq, dk, dv), (mq, mk, mv)
