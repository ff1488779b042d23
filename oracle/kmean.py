"""Windowed channel-mean removal for keys (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

Sec. 4.2: keys remove a windowed channel-wise mean after rotation (Tab. 1 shows
why: rotation alone leaves a channel mean that a token-level offset cannot
absorb); App. B adds that the mean is kept in INT8.

Readings
--------
* M1 windows are W = 128 consecutive tokens, aligned to token 0 (the same
  length as the BF16 residual window of Sec. 5.1; with n = 1024 it makes the
  2.68 bits-per-value storage figure exact).
* M2 the mean of channel j over a window is the left-to-right fp64 sum of the
  rotated values divided by W.
* M3 INT8: symmetric, one fp16 scale per (window, head):
  s = fp16(fp32(max_j |mu_j| / 127)); q_j = clamp(rint(mu_j / s), -127, 127)
  (0 when s = 0); the encoder subtracts the dequantized mean s * q_j, so the
  decoder and the encoder use the same mean.
"""

from __future__ import annotations

import numpy as np


def window_mean(y: np.ndarray) -> np.ndarray:
    """mu over axis -2 (tokens) of y[..., W, d]: sequential fp64 sum / W (M2)."""
    W = y.shape[-2]
    acc = np.zeros(y.shape[:-2] + (y.shape[-1],), dtype=np.float64)
    for t in range(W):
        acc = acc + y[..., t, :]
    return acc / float(W)


def quantize_mean(mu: np.ndarray):
    """(q int8 [..., d], scale fp16 [...]) for mu[..., d] (reading M3)."""
    amax = np.max(np.abs(mu), axis=-1)
    scale = (amax / 127.0).astype(np.float32).astype(np.float16)
    s64 = scale.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(s64[..., None] > 0, mu / np.where(s64 > 0, s64, 1.0)[..., None], 0.0)
    q = np.clip(np.rint(ratio), -127, 127).astype(np.int8)
    return q, scale


def dequantize_mean(q: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """mu_hat_j = s * q_j in fp64 (exact)."""
    return scale.astype(np.float64)[..., None] * q.astype(np.float64)
