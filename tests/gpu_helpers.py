"""Helpers for the GPU parity tests: uploading seeded inputs, the tolerance
check, sampled row selection."""
from __future__ import annotations

import sys

import numpy as np
import torch

# max |gpu - oracle| <= TOL * RMS(oracle output over the compared elements)
TOL = {"f32": 1e-4, "bf16": 2e-2}
# max |lse_gpu - lse_oracle| (natural log). Both kernels form the row sum l
# from the fp32 values of P (the bf16 kernel rounds P to bf16 only as the
# operand of P V), and the inputs are the same values on both sides, so the
# log-sum-exp differs from the oracle's by fp32 rounding of the logits, exp2
# and the sums: 1e-4 covers it for either dtype.
LSE_ATOL = {"f32": 1e-4, "bf16": 1e-4}


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(arr_f32, bits=None, dtype="f32", device="cuda"):
    """Upload fp32 values, or the bf16 bit patterns when given."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr_f32, dtype=np.float32))
    return t.to(device)


def chunk_to_dev(d, dtype):
    return tuple(to_dev(d[n], d.get(n + "_bits"), dtype) for n in "qkv")


def from_dev(t):
    return t.float().cpu().numpy()


def assert_close(got, want, dtype, what=""):
    """max |got - want| <= TOL[dtype] * RMS(want), RMS over the compared elements."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    rms = float(np.sqrt(np.mean(want ** 2)))
    err = float(np.max(np.abs(got - want)))
    tol = TOL[dtype] * rms
    say(f"  {what}: max|err| = {err:.3e}, rms = {rms:.3e}, ratio = {err / rms:.2e} (tol {TOL[dtype]:.0e})")
    assert err <= tol, f"{what}: max|err| {err:.3e} > {tol:.3e} ({TOL[dtype]} x rms {rms:.3e})"


def assert_rounds_to(o_bf16, o_f32, what=""):
    """The bf16 output of a kernel is its fp32 output (the ``_f32out`` entry
    point: same arithmetic, no final rounding) rounded to nearest even, bit
    for bit. With this, holding the fp32 output to the bf16 bar holds the
    kernel's arithmetic to it, and the bf16 output differs from that only by
    the rounding of its own format (up to 2^-9 of each value)."""
    assert o_bf16.dtype == torch.bfloat16 and o_f32.dtype == torch.float32
    rounded = o_f32.to(torch.bfloat16).view(torch.int16)
    diff = int((rounded != o_bf16.view(torch.int16)).sum())
    say(f"  {what}: bf16 output == RNE(fp32 output) except in {diff} of {o_bf16.numel()} elements")
    assert diff == 0, f"{what}: bf16 output is not the rounded fp32 output in {diff} elements"


def sample_rows(n: int, tile: int = 128, k: int = 96, seed: int = 0):
    """Rows to compare at large sizes: the first and last rows, both rows
    around every tile boundary near the start and end, plus random rows."""
    rng = np.random.default_rng(seed)
    rows = {0, 1, n - 1, n - 2}
    for b in list(range(tile, min(n, 4 * tile), tile)) + list(range((n // tile) * tile, 0, -tile))[:3]:
        rows.update({b - 1, b})
    rows.update(rng.choice(n, size=min(k, n), replace=False).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < n))
