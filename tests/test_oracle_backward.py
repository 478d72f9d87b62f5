"""Pins of the backward oracle (``oracle.backward``).

The paper prints no gradients, so the oracle is pinned by what the
mathematics fixes: central finite differences of the forward oracle (the
loss sum(O * dO)), PyTorch's CPU autograd through scaled_dot_product_attention
with an explicit boolean mask, the closed forms sum_j dK_j = 0 (softmax is
invariant to a shift of all of a row's logits) and sum_j dV_j = sum_i dO_i
(rows of P sum to one), and the locality of the chunk pattern (a chunk's dQ
does not see keys outside its allowed set; a key chunk's dK/dV does not see
queries that cannot attend to it). Planted mistakes must fail a pin.
"""
import math

import numpy as np
import pytest
import torch

import oracle.backward as bwd
from oracle import ChunkGeometry, allowed_mask, masked_attention
from oracle.attention import chunk_start


def _case(seed, g, frames, D=4, B=1, H=1):
    rng = np.random.default_rng(seed)
    L = frames * g.tokens_per_frame
    return [rng.standard_normal((B, L, H, D)) for _ in range(4)], L


def _loss(q, k, v, do, mask, scale):
    o, _ = masked_attention(q, k, v, mask, scale, dtype=np.float64)
    return float((o * do).sum())


def test_gradients_match_central_differences():
    g = ChunkGeometry(2, 2, 1, 1)
    (q, k, v, do), L = _case(1, g, 5, D=3)
    q, k, v, do = (x[0, :, 0] for x in (q, k, v, do))
    pos = np.arange(L)
    mask = allowed_mask(pos, pos, g)
    scale = 0.7
    dq, dk, dv = bwd.masked_attention_backward(q, k, v, do, mask, scale)
    eps = 1e-6
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            num[idx] = (_loss(args_p["q"], args_p["k"], args_p["v"], do, mask, scale)
                        - _loss(args_m["q"], args_m["k"], args_m["v"], do, mask, scale)) / (2 * eps)
        assert np.allclose(grad, num, rtol=1e-6, atol=1e-8), name


def test_gradients_match_torch_autograd():
    for (T, C, R, W, frames) in ((3, 2, 1, 1, 8), (2, 3, 3, 0, 11), (4, 1, 1, 2, 7)):
        g = ChunkGeometry(T, C, R, W)
        (q, k, v, do), L = _case(T + C + W, g, frames, D=8, B=2, H=2)
        dq, dk, dv = bwd.full_sequence_attention_backward(q, k, v, do, g)
        pos = np.arange(L)
        mask = torch.from_numpy(allowed_mask(pos, pos, g))
        tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3).clone().requires_grad_(True)
                      for x in (q, k, v))
        o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
        o.backward(torch.from_numpy(do).permute(0, 2, 1, 3))
        for mine, t in ((dq, tq), (dk, tk), (dv, tv)):
            assert np.allclose(mine, t.grad.permute(0, 2, 1, 3).numpy(), rtol=1e-10, atol=1e-12)


def test_closed_forms_of_key_sums():
    g = ChunkGeometry(5, 2, 1, 1)
    (q, k, v, do), L = _case(3, g, 9, D=6, B=1, H=3)
    dq, dk, dv = bwd.full_sequence_attention_backward(q, k, v, do, g)
    assert np.allclose(dk.sum(axis=1), 0.0, atol=1e-11)
    assert np.allclose(dv.sum(axis=1), do.sum(axis=1), atol=1e-11)


def test_gradients_respect_the_chunk_pattern():
    g = ChunkGeometry(3, 2, 1, 1)
    (q, k, v, do), L = _case(4, g, 9, D=4)
    base = bwd.full_sequence_attention_backward(q, k, v, do, g)
    # query chunk 3 sees c_0, c_2 and c_3
    a = 3
    lo, hi = chunk_start(a, g), chunk_start(a + 1, g)
    k2, v2 = k.copy(), v.copy()
    c1 = slice(chunk_start(1, g), chunk_start(2, g))  # chunk 1: not seen by chunk 3
    k2[:, c1] += 50.0
    v2[:, c1] -= 30.0
    pert = bwd.full_sequence_attention_backward(q, k2, v2, do, g)
    assert np.array_equal(pert[0][:, lo:hi], base[0][:, lo:hi])       # dQ of chunk 3 unchanged
    # key chunk 1 is seen by query chunks 1 and 2 only: Q/dO of chunk 3 do not reach its dK/dV
    q3, do3 = q.copy(), do.copy()
    q3[:, lo:hi] *= 7.0
    do3[:, lo:hi] += 5.0
    pert = bwd.full_sequence_attention_backward(q3, k, v, do3, g)
    for i in (1, 2):
        assert np.array_equal(pert[i][:, c1], base[i][:, c1])


# --------------------------------------------------------------------------- planted mistakes


def _pins_hold():
    try:
        test_gradients_match_torch_autograd()
        test_closed_forms_of_key_sums()
    except AssertionError:
        return False
    return True


def test_unmutated_backward_oracle_passes():
    assert _pins_hold()


def _mutant(kind):
    def f(q, k, v, do, mask, scale, *, dtype=np.float64, magnitudes=False):
        q, k, v, do = (np.asarray(x, dtype=dtype) for x in (q, k, v, do))
        s = np.where(mask, (q @ k.T) * scale, -np.inf)
        e = np.where(mask, np.exp(s - s.max(axis=1, keepdims=True)), 0.0)
        p = e / e.sum(axis=1, keepdims=True)
        dv = (p @ do) if kind == "dv_untransposed" else (p.T @ do)
        dp = do @ v.T
        ds = p * dp if kind == "ds_no_rowsum" else p * (dp - (p * dp).sum(axis=1, keepdims=True))
        dq = (ds @ k) if kind == "dq_no_scale" else scale * (ds @ k)
        dk = scale * ((ds @ q) if kind == "dk_untransposed" else (ds.T @ q))
        return dq, dk, dv
    return f


@pytest.mark.parametrize("kind", ["dv_untransposed", "ds_no_rowsum", "dq_no_scale", "dk_untransposed"])
def test_backward_mutants_fail_a_pin(monkeypatch, kind):
    monkeypatch.setattr(bwd, "masked_attention_backward", _mutant(kind))
    assert not _pins_hold()


def test_magnitudes_bound_the_gradients():
    # |sum x y| <= sum |x y|, with equality when all products share a sign
    g = ChunkGeometry(4, 2, 1, 1)
    (q, k, v, do), L = _case(9, g, 7, D=5, B=1, H=2)
    grads, mags = bwd.full_sequence_attention_backward(q, k, v, do, g, magnitudes=True)
    plain = bwd.full_sequence_attention_backward(q, k, v, do, g)
    for gr, pl, mg in zip(grads, plain, mags):
        assert np.array_equal(gr, pl)
        assert np.all(np.abs(gr) <= mg * (1 + 1e-12) + 1e-300)
    pos = np.arange(L)
    mask = allowed_mask(pos, pos, g)
    ones = np.ones((L, 5))
    _, (_, _, mdv) = bwd.masked_attention_backward(q[0, :, 0], k[0, :, 0], v[0, :, 0], ones, mask, 0.5,
                                                   magnitudes=True)
    dq, dk, dv = bwd.masked_attention_backward(q[0, :, 0], k[0, :, 0], v[0, :, 0], ones, mask, 0.5)
    assert np.allclose(mdv, dv)  # dO = 1 > 0: |P|^T |dO| = P^T dO


# --------------------------------------------------------------------------- magnitudes, pinned from both sides

_MAG_CASES = ((3, 2, 1, 1, 7, 4), (2, 3, 3, 0, 9, 3), (4, 1, 1, 2, 6, 5))


def _magnitudes_match_brute_force():
    """The oracle's gradients and absolute-product sums against the fp64
    element loop of ``oracle.brute`` (a second construction: key sets as
    Python sets, per-element math.fsum)."""
    from oracle.brute import brute_force_backward
    for (T, C, R, W, frames, D) in _MAG_CASES:
        g = ChunkGeometry(T, C, R, W)
        (q, k, v, do), L = _case(T * 7 + W, g, frames, D=D)
        (bg, bm) = brute_force_backward(q[0, :, 0], k[0, :, 0], v[0, :, 0], do[0, :, 0],
                                        T=T, C=C, R=R, W=W)
        grads, mags = bwd.full_sequence_attention_backward(q, k, v, do, g, magnitudes=True)
        for mine, ref in zip(grads + mags, bg + bm):
            if not np.allclose(mine[0, :, 0], ref, rtol=1e-12, atol=1e-14):
                return False
    return True


def test_magnitudes_match_brute_force():
    assert _magnitudes_match_brute_force()


def _magnitude_mutant(kind):
    real = bwd.masked_attention_backward

    def f(q, k, v, do, mask, scale, *, dtype=np.float64, magnitudes=False):
        grads = real(q, k, v, do, mask, scale, dtype=dtype)
        if not magnitudes:
            return grads
        q, k, v, do = (np.asarray(x, dtype=dtype) for x in (q, k, v, do))
        s = np.where(mask, (q @ k.T) * scale, -np.inf)
        e = np.where(mask, np.exp(s - s.max(axis=1, keepdims=True)), 0.0)
        p = e / e.sum(axis=1, keepdims=True)
        dp = do @ v.T
        ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
        a = np.abs(dp * p) if kind == "abs_dp_for_ds" else np.abs(ds)
        sq = 1.0 if kind == "scale_dropped" else scale
        mq = sq * (a @ np.abs(k))
        mk = sq * ((a @ np.abs(q)) if kind == "untransposed_dk" else (a.T @ np.abs(q)))
        mv = (p.T @ do) if kind == "dv_no_abs" else (p.T @ np.abs(do))
        return grads, (mq, mk, mv)
    return f


@pytest.mark.parametrize("kind", ["scale_dropped", "abs_dp_for_ds", "untransposed_dk", "dv_no_abs"])
def test_magnitude_mutants_fail_the_brute_force_pin(monkeypatch, kind):
    monkeypatch.setattr(bwd, "masked_attention_backward", _magnitude_mutant(kind))
    assert not _magnitudes_match_brute_force()


def test_sampled_backward_equals_the_full_oracle():
    """Row blocks and selected rows change nothing: the sampled form equals the
    full-matrix oracle on the rows it returns (ragged blocks of 7 rows, two
    batch elements, a subset of heads, W = 1 and W = 2)."""
    for (T, C, R, W, frames) in ((5, 2, 1, 1, 9), (3, 2, 3, 2, 12)):
        g = ChunkGeometry(T, C, R, W)
        (q, k, v, do), L = _case(31 + W, g, frames, D=6, B=2, H=3)
        grads, mags = bwd.full_sequence_attention_backward(q, k, v, do, g, heads=[0, 2],
                                                           magnitudes=True)
        rng = np.random.default_rng(W)
        qr = np.unique(np.r_[0, L - 1, rng.choice(L, 9, replace=False)])
        kr = np.unique(np.r_[0, L - 1, rng.choice(L, 9, replace=False)])
        sg, sm = bwd.sampled_sequence_attention_backward(q, k, v, do, g, q_rows=qr, k_rows=kr,
                                                         heads=[0, 2], row_block=7)
        for i, (full, part) in enumerate(zip(grads + mags, sg + sm)):
            rows = qr if i % 3 == 0 else kr
            assert np.allclose(full[:, rows], part, rtol=1e-12, atol=1e-14), i
