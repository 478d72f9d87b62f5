"""Planted mistakes in the oracle must fail at least one pin.

Each mutant below is a plausible slip in the oracle (a dropped c_0 term, a
window off by one, a transposed operand, a wrong sign, an unnormalised row);
the pin checks used in ``test_oracle`` are rerun against the mutant and must
reject it. Mistakes are planted on the CPU only.
"""
import math

import numpy as np
import pytest

import oracle.attention as att
import oracle.geometry as geo
from oracle import ChunkGeometry, brute_force_attention


def _pins_hold():
    """A compact rerun of the brute-force, pair-count and zero-Q pins."""
    T, C, R, W, frames, D = 3, 2, 1, 1, 8, 8
    L = T * frames
    rng = np.random.default_rng(123)
    q, k, v = (rng.standard_normal((L, D)).astype(np.float32) for _ in range(3))
    g = ChunkGeometry(T, C, R, W)
    pos = np.arange(L)
    mask = geo.allowed_mask(pos, pos, g)
    o, lse = att.masked_attention(q, k, v, mask, 1 / math.sqrt(D), dtype=np.float64)
    bo, blse, _ = brute_force_attention(q, k, v, T=T, C=C, R=R, W=W)
    ok = np.allclose(o, bo, atol=1e-10) and np.allclose(lse, blse, atol=1e-10)
    closed = 64 * 64 + 128 * 192 + 3 * 128 * 320
    ok &= geo.allowed_pair_count(9 * 64, ChunkGeometry(64, 2, 1, 1)) == closed
    return bool(ok)


def test_unmutated_oracle_passes():
    assert _pins_hold()


def _mask_without_c0(q_pos, k_pos, g):
    a = geo.chunk_of_position(q_pos, g)[:, None]
    c = geo.chunk_of_position(k_pos, g)[None, :]
    return (c >= a - g.window) & (c <= a)


def _mask_window_plus_one(q_pos, k_pos, g):
    a = geo.chunk_of_position(q_pos, g)[:, None]
    c = geo.chunk_of_position(k_pos, g)[None, :]
    return (c == 0) | ((c >= a - g.window - 1) & (c <= a))


def _mask_strictly_causal_inside_chunk(q_pos, k_pos, g):
    base = (lambda a, c: (c == 0) | ((c >= a - g.window) & (c <= a)))(
        geo.chunk_of_position(q_pos, g)[:, None], geo.chunk_of_position(k_pos, g)[None, :])
    return base & (np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None])


def _attn_transposed(q, k, v, mask, scale, *, dtype=np.float32, return_probs=False):
    # logits transposed: S^T = K Q^T used as if it were S (square case)
    s = (np.asarray(k, dtype) @ np.asarray(q, dtype).T) * dtype(scale)
    s = np.where(mask, s, -np.inf)
    m = s.max(1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(1, keepdims=True)
    p = np.where(mask, e / z, 0)
    return p @ np.asarray(v, dtype), m[:, 0] + np.log(z[:, 0])


def _attn_wrong_sign(q, k, v, mask, scale, *, dtype=np.float32, return_probs=False):
    s = -(np.asarray(q, dtype) @ np.asarray(k, dtype).T) * dtype(scale)
    s = np.where(mask, s, -np.inf)
    m = s.max(1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(1, keepdims=True)
    p = np.where(mask, e / z, 0)
    return p @ np.asarray(v, dtype), m[:, 0] + np.log(z[:, 0])


def _attn_unnormalised(q, k, v, mask, scale, *, dtype=np.float32, return_probs=False):
    s = (np.asarray(q, dtype) @ np.asarray(k, dtype).T) * dtype(scale)
    s = np.where(mask, s, -np.inf)
    m = s.max(1, keepdims=True)
    e = np.where(mask, np.exp(s - m), 0)
    return e @ np.asarray(v, dtype), m[:, 0] + np.log(e.sum(1))


@pytest.mark.parametrize("target,name,mutant", [
    (geo, "allowed_mask", _mask_without_c0),
    (geo, "allowed_mask", _mask_window_plus_one),
    (geo, "allowed_mask", _mask_strictly_causal_inside_chunk),
    (att, "masked_attention", _attn_transposed),
    (att, "masked_attention", _attn_wrong_sign),
    (att, "masked_attention", _attn_unnormalised),
])
def test_planted_mistake_is_caught(monkeypatch, target, name, mutant):
    monkeypatch.setattr(target, name, mutant)
    assert not _pins_hold()


# --------------------------------------------------------------------------- producer mutants


def _producer_pins_hold(fn):
    """The unit-RMS, closed-form and torch pins of ``test_oracle`` against fn."""
    import torch
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 5, 3, 64)) * rng.uniform(0.5, 4.0, size=(2, 5, 3, 1))
    g = rng.uniform(0.5, 1.5, size=(3, 64))
    y = fn(x)
    ok = np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, atol=1e-10)
    ok &= np.allclose(fn(np.full((1, 1, 3, 64), 2.0), None, eps=5.0), 2.0 / 3.0)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), eps=1e-6).numpy() * g
    ok &= np.allclose(fn(x, g, 1e-6), ref, atol=1e-10)
    return bool(ok)


def _rms_over_heads(x, gain=None, eps=0.0):
    x = np.asarray(x, dtype=np.float64)
    y = x / np.sqrt(np.mean(x * x, axis=(-2, -1), keepdims=True) + eps)  # wrong group
    return y * gain if gain is not None else y


def _rms_eps_outside(x, gain=None, eps=0.0):
    x = np.asarray(x, dtype=np.float64)
    y = x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps)  # eps after the root
    return y * gain if gain is not None else y


def _rms_no_root(x, gain=None, eps=0.0):
    x = np.asarray(x, dtype=np.float64)
    y = x / (np.mean(x * x, axis=-1, keepdims=True) + eps)  # mean square, not its root
    return y * gain if gain is not None else y


def test_unmutated_producer_oracle_passes():
    from oracle import rms_normalise
    assert _producer_pins_hold(rms_normalise)


@pytest.mark.parametrize("mutant", [_rms_over_heads, _rms_eps_outside, _rms_no_root],
                         ids=["group_over_heads", "eps_outside_root", "no_root"])
def test_producer_mutants_fail_a_pin(mutant):
    assert not _producer_pins_hold(mutant)
