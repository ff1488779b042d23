"""Seeded synthetic workloads shared by the tests, the bench and the CPU oracle.

This module holds no arithmetic of the method: only shapes, coding
parameters and random inputs.  Inputs stand in for the paper's captured
Qwen3-8B / Llama-3.1-8B caches (8 KV heads, head_dim 128), which are not
available; their recipe:

* Q ~ N(0, 1), V ~ N(0, 1).
* K[b, t, h, c] = mu[h, c] + sigma[h, c] * z with mu ~ N(0, 2) (variance 2),
  sigma ~ U(0.5, 2), and a few outlier channels per head (drawn without
  replacement) whose sigma is multiplied by 8.  mu and sigma are shared by all
  sequences and tokens.
* Everything is drawn in fp32 and rounded to bf16 (round to nearest even).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np
import torch

HEAD_DIM = 128
MEAN_WINDOW = 128
PRECISION = 12


@dataclass(frozen=True)
class Coding:
    """Coding parameters of one tensor (K or V); n values per stream."""
    levels: int
    record_bytes: int
    alpha: float
    precision: int = PRECISION
    n: int = HEAD_DIM

    @property
    def bits_per_elem(self) -> float:
        return 8.0 * self.record_bytes / self.n


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    context: int
    q_heads: int
    kv_heads: int
    outliers: int
    k: Coding
    v: Coding
    head_dim: int = HEAD_DIM
    streams: str = "head"        # "head": one stream per (token, KV head); "token": per token

    @property
    def gqa(self) -> int:
        return self.q_heads // self.kv_heads

    def with_context(self, context: int, batch: int | None = None) -> "Workload":
        return replace(self, context=context, batch=self.batch if batch is None else batch)


def record_bytes(bits_per_elem: float, n: int = HEAD_DIM) -> int:
    return int(math.floor(bits_per_elem * n / 8.0 + 1e-9))


# Level counts.  "paper": alpha = 1.4 (Sec. 5.1) and the level count with the
# lowest reconstruction error that fits the record, chosen as in Tab. 2
# (tests/golden/level_sweep.txt, written by tests/golden/make_level_sweep.py).
# "literal": the level count stated for the workload with alpha raised to the
# smallest value on a 0.1 grid that makes it fit (the stated count does not fit
# at alpha = 1.4; Tab. 2 marks such pairs as infeasible).
PAPER_LEVELS = {32: 5, 36: 6, 48: 9, 64: 17}
LITERAL_ALPHA = {(16, 32): 8.6, (16, 36): 5.6, (32, 48): 7.6, (64, 64): 7.8}


def coding(levels: int, bpe: float, variant: str) -> Coding:
    C = record_bytes(bpe)
    if variant == "paper":
        return Coding(levels=PAPER_LEVELS[C], record_bytes=C, alpha=1.4)
    if variant == "literal":
        return Coding(levels=levels, record_bytes=C, alpha=LITERAL_ALPHA[(levels, C)])
    raise ValueError(variant)


def workload(name: str, variant: str = "paper", bpe: float | None = None) -> Workload:
    """The five workloads the path is measured on, by name."""
    if name == "b1_t4k":
        c = coding(16, 2.25, variant)
        return Workload(name, 1, 4096, 32, 8, 4, c, c)
    if name == "b16_t32k":
        c = coding(16, 2.26, variant)
        return Workload(name, 16, 32768, 32, 8, 4, c, c)
    if name == "b1_t128k":
        bpe = 2.26 if bpe is None else bpe
        lv = {2.0: 16, 2.26: 16, 3.0: 32, 4.0: 64}[bpe]
        c = coding(lv, bpe, variant)
        return Workload(name, 1, 131072, 32, 8, 4, c, c)
    if name == "b64_t8k":
        c = coding(16, 2.26, variant)
        return Workload(name, 64, 8192, 32, 8, 4, c, c)
    if name == "b32_t32k_g8":
        return Workload(name, 32, 32768, 64, 8, 8, coding(32, 3.0, variant), coding(16, 2.0, variant))
    if name in TOKEN_WORKLOADS:
        # the paper's default operating point (Sec. 5.1): one stream of 1024
        # values per token, 331 B / 231 B containers (+ the 4-byte s, o header)
        # with 8 / 6 levels at alpha 1.4, and the 2^8-entry table of Sec. 3
        k, v = Coding(8, 335, 1.4, precision=8, n=1024), Coding(6, 235, 1.4, precision=8, n=1024)
        if name == "b32_t32k_g8_tok":
            # the wide-GQA shape (64 query / 8 KV heads, 8 outlier channels per
            # key head) with the per-token coding
            return Workload(name, 32, 32768, 64, 8, 8, k, v, streams="token")
        B, T = {"b1_t4k_tok": (1, 4096), "b16_t32k_tok": (16, 32768)}[name]
        return Workload(name, B, T, 32, 8, 4, k, v, streams="token")
    raise KeyError(name)


WORKLOADS = ("b1_t4k", "b16_t32k", "b1_t128k", "b64_t8k", "b32_t32k_g8")
TOKEN_WORKLOADS = ("b1_t4k_tok", "b16_t32k_tok", "b32_t32k_g8_tok")


def key_stats(seed: int, heads: int, d: int, outliers: int):
    """Per-channel (mu, sigma) of the synthetic keys, fp32 numpy [H, d]."""
    rng = np.random.default_rng(seed + 7919)
    mu = rng.normal(0.0, math.sqrt(2.0), size=(heads, d)).astype(np.float32)
    sigma = rng.uniform(0.5, 2.0, size=(heads, d)).astype(np.float32)
    for h in range(heads):
        idx = rng.choice(d, size=outliers, replace=False)
        sigma[h, idx] *= 8.0
    return mu, sigma


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_q(wl: Workload, seed: int, device="cpu", batch: int | None = None) -> torch.Tensor:
    B = wl.batch if batch is None else batch
    g = _gen(seed * 3 + 1, device)
    q = torch.randn((B, wl.q_heads, wl.head_dim), generator=g, device=device, dtype=torch.float32)
    return q.to(torch.bfloat16)


def make_k(wl: Workload, seed: int, device="cpu", batch: int | None = None,
           context: int | None = None) -> torch.Tensor:
    """Keys [B, T, H_kv, d] bf16."""
    B = wl.batch if batch is None else batch
    T = wl.context if context is None else context
    mu, sigma = key_stats(seed, wl.kv_heads, wl.head_dim, wl.outliers)
    g = _gen(seed * 3 + 2, device)
    z = torch.randn((B, T, wl.kv_heads, wl.head_dim), generator=g, device=device, dtype=torch.float32)
    mu_t = torch.from_numpy(mu).to(device)
    sg_t = torch.from_numpy(sigma).to(device)
    z.mul_(sg_t).add_(mu_t)
    return z.to(torch.bfloat16)


def make_v(wl: Workload, seed: int, device="cpu", batch: int | None = None,
           context: int | None = None) -> torch.Tensor:
    """Values [B, T, H_kv, d] bf16."""
    B = wl.batch if batch is None else batch
    T = wl.context if context is None else context
    g = _gen(seed * 3 + 3, device)
    v = torch.randn((B, T, wl.kv_heads, wl.head_dim), generator=g, device=device, dtype=torch.float32)
    return v.to(torch.bfloat16)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


# Degenerate inputs: each (token, KV head) vector takes one of these patterns.
#   zero       all channels 0 (e.g. a padding token)
#   onehot0    one non-zero channel, channel 0
#   const      every channel the same value
#   onehot     one non-zero channel, a random channel other than 0, random sign
#   twolevel   a base value, with the next bf16 value up on a random subset
#   tiny       one non-zero channel of magnitude about 1e-6
#   normal     N(0, 1) channels
EDGE_KINDS = ("zero", "onehot0", "const", "onehot", "twolevel", "tiny", "normal")


def _edge_vector(kind: str, rng: np.random.Generator, d: int, mag: float) -> np.ndarray:
    v = np.zeros(d, dtype=np.float32)
    if kind == "onehot0":
        v[0] = mag
    elif kind == "const":
        v[:] = mag
    elif kind == "onehot":
        v[1 + rng.integers(d - 1)] = mag * rng.choice([-1.0, 1.0])
    elif kind == "twolevel":
        bits = torch.tensor([mag], dtype=torch.float32).to(torch.bfloat16).view(torch.int16)
        lo = float(bits.view(torch.bfloat16).float()[0])
        hi = float((bits + 1).view(torch.bfloat16).float()[0])     # the next bf16 value up
        v[:] = lo
        v[rng.random(d) < 0.5] = hi
    elif kind == "tiny":
        v[rng.integers(d)] = np.float32(1e-6 * mag)
    elif kind == "normal":
        v[:] = rng.normal(size=d)
    elif kind != "zero":
        raise ValueError(kind)
    return v


def make_edge(seed: int, batch: int, context: int, kv_heads: int, head_dim: int = HEAD_DIM,
              kinds=EDGE_KINDS, same_heads: bool = False) -> torch.Tensor:
    """Degenerate K or V inputs [B, T, H, d] bf16: token t of head h takes
    kinds[(t + h) % len(kinds)] (kinds[t % len(kinds)] for every head when
    same_heads, with one magnitude per token, so that the whole token is
    one pattern), magnitudes drawn from U(0.25, 4)."""
    rng = np.random.default_rng(seed + 104729)
    out = np.zeros((batch, context, kv_heads, head_dim), dtype=np.float32)
    for b in range(batch):
        for t in range(context):
            mag = float(rng.uniform(0.25, 4.0))
            for h in range(kv_heads):
                kind = kinds[(t if same_heads else t + h) % len(kinds)]
                out[b, t, h] = _edge_vector(kind, rng, head_dim, mag if same_heads else float(rng.uniform(0.25, 4.0)))
    return torch.from_numpy(out).to(torch.bfloat16)


def make_edge_keys(seed: int, batch: int, context: int, kv_heads: int, head_dim: int = HEAD_DIM) -> torch.Tensor:
    """Degenerate keys [B, T, H, d] bf16, one pattern per 128-token window
    (cycling): every token 127 e_0; every token 0; every token the same
    N(0, 1) vector (a token equal to its window's mean); the mixed patterns of
    make_edge."""
    if context % MEAN_WINDOW:
        raise ValueError("context must be a multiple of the mean window")
    mixed = make_edge(seed, batch, context, kv_heads, head_dim).float().numpy()
    rng = np.random.default_rng(seed + 15485863)
    out = np.zeros((batch, context, kv_heads, head_dim), dtype=np.float32)
    for w in range(context // MEAN_WINDOW):
        sl = slice(w * MEAN_WINDOW, (w + 1) * MEAN_WINDOW)
        kind = w % 4
        if kind == 0:
            out[:, sl, :, 0] = 127.0
        elif kind == 2:
            out[:, sl] = rng.normal(size=(batch, 1, kv_heads, head_dim)).astype(np.float32)
        elif kind == 3:
            out[:, sl] = mixed[:, sl]
    return torch.from_numpy(out).to(torch.bfloat16)


def make_ternary(seed: int, batch: int, context: int, kv_heads: int, head_dim: int = HEAD_DIM) -> torch.Tensor:
    """K or V inputs [B, T, H, d] bf16 with every channel in {-1, 0, 1}
    (probabilities 1/4, 1/2, 1/4): the sums and differences of up to 128 such
    values are integers below 256, which bf16 holds exactly."""
    rng = np.random.default_rng(seed + 1299709)
    v = rng.choice(np.array([-1.0, 0.0, 0.0, 1.0], dtype=np.float32), size=(batch, context, kv_heads, head_dim))
    return torch.from_numpy(v).to(torch.bfloat16)
