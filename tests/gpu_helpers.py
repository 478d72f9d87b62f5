"""Helpers for the GPU parity tests: uploading seeded inputs, the tolerance
check, sampled row selection."""
from __future__ import annotations

import sys

import numpy as np
import torch

# max |gpu - oracle| <= TOL * RMS(oracle output over the compared elements)
TOL = {"f32": 1e-4, "bf16": 2e-2}


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


def assert_close(got, want, dtype, what="", output_rounding=False):
    """max |got - want| <= TOL[dtype] * RMS(want).

    ``output_rounding`` (bf16 only) adds, element by element, the largest
    error of rounding the exact value to a bf16 output, 2^-8 |want|: used for
    small edge-case geometries whose queries see few keys, where |o| reaches
    many times its RMS and that rounding alone can exceed 2e-2 x RMS.
    """
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    rms = float(np.sqrt(np.mean(want ** 2)))
    diff = np.abs(got - want)
    err = float(np.max(diff))
    tol = TOL[dtype] * rms
    if output_rounding and dtype == "bf16":
        worst = float(np.max(diff / (tol + 2.0 ** -8 * np.abs(want))))
        say(f"  {what}: max|err| = {err:.3e}, rms = {rms:.3e}, ratio = {err / rms:.2e}, "
            f"worst err / (2e-2 rms + 2^-8 |o|) = {worst:.3f}")
        assert worst <= 1.0, f"{what}: error {worst:.3f} x the rounding-aware bound"
        return
    say(f"  {what}: max|err| = {err:.3e}, rms = {rms:.3e}, ratio = {err / rms:.2e} (tol {TOL[dtype]:.0e})")
    assert err <= tol, f"{what}: max|err| {err:.3e} > {tol:.3e} ({TOL[dtype]} x rms {rms:.3e})"


def sample_rows(n: int, tile: int = 128, k: int = 96, seed: int = 0):
    """Rows to compare at large sizes: the first and last rows, both rows
    around every tile boundary near the start and end, plus random rows."""
    rng = np.random.default_rng(seed)
    rows = {0, 1, n - 1, n - 2}
    for b in list(range(tile, min(n, 4 * tile), tile)) + list(range((n // tile) * tile, 0, -tile))[:3]:
        rows.update({b - 1, b})
    rows.update(rng.choice(n, size=min(k, n), replace=False).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < n))
