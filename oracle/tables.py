"""Calibration-free entropy model and budget arithmetic (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

What the paper fixes
--------------------
* Sec. 4.2: after rotation and mean removal each stream is quantized on a
  token-wise min-max grid with M levels; the entropy model comes from Gaussian
  order statistics, and because normalized positions are affine invariant one
  table serves every token and layer.
* Sec. 4.4 (distribution sharpening): p'_m is proportional to p_m ** alpha.
* Sec. 3.1, Eq. (rans): integer frequencies f_m with sum 2**p, cumulative c_m.
* Alg. 1: r_m = -log2(f_m / sum f); Eq. (budget): B = 8 C - sigma.

Readings (the paper is silent or loose here)
--------------------------------------------
* T1 the entropy model from order statistics of normal samples (Sec. 4.2):
  the min and max of a stream of n standard normals are replaced by their expectations -a_n and +a_n, with
  a_n = E[max of n iid N(0,1)].  Level m then covers the interval between the
  edges e_m = a_n((2m-1)/(M-1) - 1) and e_{m+1} (e_0 = -inf, e_M = +inf), and
  its probability is the normal CDF mass between them.  Only the lower half is
  computed; the upper half is its mirror, so the table is exactly symmetric.
* T2 quantization to 2**p: symmetric largest-remainder apportionment over the
  lower half (ties in the fractional part go to the lower m), every f_m >= 1,
  mirrored; an odd M gives its centre symbol what is left.
* T3 costs are carried as Q16 integers R_m = round(2**16 (p - log2 f_m)) so
  that the budget test sum R <= B_Q16 is exact and order free.
* T4 a record of C bytes holds the fp16 scale and offset (4 bytes) followed by
  the paper's container: the 32-bit final state (sigma = 32) and the renorm
  bytes.  So B = 8 (C - 4) - 32 bits.  With n = 1024 this reproduces the paper's
  storage figures (331 B container + 4 B metadata + 8 B of INT8 mean per token
  for keys gives 2.68 bits per value, 231 + 4 B gives 1.84).
* T5 the Lagrange multiplier grid: lambda = 2**(U/512) for integer U, held as
  fp32 values Lambda[k] = 2**(k/512), k in [0, 512) scaled by 2**floor(U/512).
"""

from __future__ import annotations

import math
import warnings
from dataclasses import dataclass

import numpy as np
from scipy import integrate, special

Q16 = 1 << 16
LAMBDA_STEPS = 512          # grid points per octave of lambda (reading T5)
SIGMA_BITS = 32             # final rANS state, written as 4 bytes (reading T4)
HEADER_BYTES = 4            # fp16 scale + fp16 offset (reading T4)


def normal_cdf(x):
    """Phi(x) = erfc(-x / sqrt 2) / 2, accurate in both tails."""
    return 0.5 * special.erfc(-np.asarray(x, dtype=np.float64) / math.sqrt(2.0))


def expected_max_normal(n: int) -> float:
    """a_n = E[max of n iid standard normals] (reading T1).

    a_n = integral of x * n * phi(x) * Phi(x)**(n-1) over the real line.
    """
    if n < 1:
        raise ValueError("n must be >= 1")
    if n == 1:
        return 0.0

    def integrand(x):
        phi = math.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
        cdf = 0.5 * math.erfc(-x / math.sqrt(2.0))
        return x * n * phi * cdf ** (n - 1)

    total = 0.0
    # split so quad sees the peak region with fine resolution
    with warnings.catch_warnings():
        warnings.simplefilter("ignore", integrate.IntegrationWarning)
        for lo, hi in ((-40.0, -8.0), (-8.0, 0.0), (0.0, 2.0), (2.0, 4.0), (4.0, 8.0), (8.0, 40.0)):
            val, _ = integrate.quad(integrand, lo, hi, epsabs=1e-15, epsrel=1e-14, limit=400)
            total += val
    return total


def level_probabilities(n: int, M: int) -> np.ndarray:
    """Normal-CDF mass of the M levels of a min-max grid (reading T1), fp64."""
    if M < 2:
        raise ValueError("M must be >= 2")
    a = expected_max_normal(n)
    half = M // 2
    q = np.zeros(M, dtype=np.float64)
    # lower half: q_m = Phi(e_{m+1}) - Phi(e_m), e_0 = -inf
    prev = 0.0
    for m in range(half):
        edge = a * ((2.0 * (m + 1) - 1.0) / (M - 1) - 1.0)
        cur = float(normal_cdf(edge))
        q[m] = cur - prev
        prev = cur
    if M % 2 == 1:
        c = half
        # centre interval is (-a/(M-1), +a/(M-1)): mass erf(u / sqrt 2)
        q[c] = float(special.erf(a / (M - 1) / math.sqrt(2.0)))
    for m in range(half):
        q[M - 1 - m] = q[m]
    return q


def sharpen(q: np.ndarray, alpha: float) -> np.ndarray:
    """Sec. 4.4: p'_m = p_m**alpha / sum_k p_k**alpha."""
    w = np.power(q, float(alpha))
    return w / w.sum()


def quantize_frequencies(qs: np.ndarray, p: int) -> np.ndarray:
    """Integer frequencies with sum 2**p, all >= 1, exactly symmetric (T2)."""
    M = qs.shape[0]
    total = 1 << p
    half = M // 2
    g = qs[:half] * float(total)
    if M % 2 == 1:
        H = int(math.floor(float(g.sum()) + 0.5))
        H = min(H, (total - 1) // 2)
    else:
        H = total // 2
    if H < half:
        raise ValueError("precision too small for this many levels")
    f = np.maximum(1, np.floor(g)).astype(np.int64)
    deficit = H - int(f.sum())
    if deficit > 0:
        frac = g - np.floor(g)
        order = sorted(range(half), key=lambda m: (-frac[m], m))
        k = 0
        while deficit > 0:
            f[order[k % half]] += 1
            deficit -= 1
            k += 1
    while deficit < 0:
        # clamping to 1 over-allocated: take units back from the largest
        m = min(range(half), key=lambda i: (-f[i], i))
        if f[m] <= 1:
            raise ValueError("cannot apportion frequencies")
        f[m] -= 1
        deficit += 1
    full = np.zeros(M, dtype=np.int64)
    full[:half] = f
    full[M - half:] = f[::-1]
    if M % 2 == 1:
        full[half] = total - 2 * H
    assert int(full.sum()) == total and full.min() >= 1
    return full


def cost_q16(freq: np.ndarray, p: int) -> np.ndarray:
    """R_m = round(2**16 * (p - log2 f_m)) (Alg. 1 costs, reading T3)."""
    r = float(p) - np.log2(freq.astype(np.float64))
    return np.floor(r * Q16 + 0.5).astype(np.int64)


def lambda_table() -> np.ndarray:
    """Lambda[k] = fp32(2**(k/512)), k in [0, 512) (reading T5)."""
    k = np.arange(LAMBDA_STEPS, dtype=np.float64)
    return np.exp2(k / LAMBDA_STEPS).astype(np.float32)


def record_budget_q16(record_bytes: int) -> int:
    """B in Q16 bits for a C-byte record: 8 (C - 4) - sigma (Eq. budget, T4)."""
    bits = 8 * (record_bytes - HEADER_BYTES) - SIGMA_BITS
    return bits * Q16


def record_bytes_for(bits_per_elem: float, n: int) -> int:
    """C = floor(bpe * n / 8): the record covers header and container."""
    return int(math.floor(bits_per_elem * n / 8.0 + 1e-9))


@dataclass
class Tables:
    n: int
    M: int
    p: int
    alpha: float
    record_bytes: int
    freq: np.ndarray        # int64 [M]
    cum: np.ndarray         # int64 [M]
    cost: np.ndarray        # int64 [M]  (Q16)
    sym_of_z: np.ndarray    # int64 [2**p]
    lam: np.ndarray         # float32 [512]
    budget_q16: int
    feasible: bool

    @property
    def rate(self) -> np.ndarray:
        """Real-valued costs r_m = R_m * 2**-16 (exact in fp64)."""
        return self.cost.astype(np.float64) / Q16

    @property
    def cheapest(self) -> int:
        """Lowest index among the symbols of minimum cost."""
        return int(np.argmin(self.cost))


def build_tables(n: int, M: int, p: int, alpha: float, record_bytes: int) -> Tables:
    q = level_probabilities(n, M)
    qs = sharpen(q, alpha)
    freq = quantize_frequencies(qs, p)
    cum = np.concatenate([[0], np.cumsum(freq)[:-1]]).astype(np.int64)
    cost = cost_q16(freq, p)
    sym = np.repeat(np.arange(M, dtype=np.int64), freq)
    budget = record_budget_q16(record_bytes)
    feasible = bool(n * int(cost.min()) <= budget) and budget > 0
    return Tables(n=n, M=M, p=p, alpha=float(alpha), record_bytes=record_bytes,
                  freq=freq, cum=cum, cost=cost, sym_of_z=sym, lam=lambda_table(),
                  budget_q16=budget, feasible=feasible)
