"""Per-head Hadamard rotation (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

Sec. 4.2 applies a Hadamard rotation to each attention head before
quantization (keys online, values foldable into weights); Fig. 1 shows it as
the first stage of the pipeline.

Reading H1: the unnormalized Sylvester matrix H_d (entries +-1, H H^T = d I,
H symmetric), applied as the fast Walsh-Hadamard transform with stages
h = 1, 2, 4, ..., d/2, each stage replacing a pair (a, b) at positions
(i, i + h) (bit h of i clear) by (a + b, a - b).  Arithmetic is fp64; the stage
order is part of the definition so that the result is reproducible to the bit.
The inverse is H / d.
"""

from __future__ import annotations

import numpy as np


def fwht(x: np.ndarray) -> np.ndarray:
    """Unnormalized FWHT over the last axis (fp64, fixed stage order)."""
    v = np.array(x, dtype=np.float64, copy=True)
    d = v.shape[-1]
    if d & (d - 1):
        raise ValueError("head_dim must be a power of two")
    lead = v.shape[:-1]
    h = 1
    while h < d:
        w = v.reshape(*lead, d // (2 * h), 2, h)
        a = w[..., 0, :]
        b = w[..., 1, :]
        w = np.stack([a + b, a - b], axis=-2)
        v = w.reshape(*lead, d)
        h *= 2
    return v


def sylvester(d: int) -> np.ndarray:
    """Explicit Sylvester Hadamard matrix (integer), for tests."""
    H = np.ones((1, 1), dtype=np.int64)
    while H.shape[0] < d:
        H = np.block([[H, H], [H, -H]])
    return H
