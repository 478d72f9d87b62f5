"""Oracle of the fused K/V producer: RMS normalisation of the query and key
rows of a chunk before its keys and values enter the KV cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's student keeps the teacher's DiT blocks (Sec. 4.1: WAN2.1 I2V
14B), whose attention normalises queries and keys by their root mean square
before the attention equation of Sec. 4.2; the cached keys of Sec. 4.3 are
these normalised keys. The normalisation group is read as one (token, head)
row of D elements:

    y[d] = x[d] / sqrt(mean_d(x[d]^2) + eps) * gain[h, d]

computed here in float64 and returned in float64 (the caller rounds to the
output dtype when it compares).
"""
from __future__ import annotations

import numpy as np


def rms_normalise(x, gain=None, eps: float = 0.0):
    """x: [..., H, D]; gain: [H, D] or None (ones). Returns float64 [..., H, D]."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    y = x / np.sqrt(ms + eps)
    if gain is not None:
        y = y * np.asarray(gain, dtype=np.float64)
    return y
