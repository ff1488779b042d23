"""Token-wise affine grid, Drift and Refit: Alg. 1 of App. A (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

What the paper fixes
--------------------
* Eq. (affine_token): x_hat_i = o + s m_i, m_i in {0..M-1},
  s = (max x - min x)/(M - 1), o = min x.
* Eq. (drift): minimize sum_i (x_i - (o + s m_i))**2 subject to
  sum_i r(m_i) <= B, solved through Eq. (lagrangian): for a fixed lambda each
  value independently takes argmin_m D_i(m) + lambda r(m); bisection on lambda.
* Alg. 1: FitMinMax -> Drift -> Refit -> fp16(s), fp16(o) -> Drift -> rANS.
  Drift bisects log2 lambda rather than lambda (App. A) for T = 12 steps
  inside [hi - 40, hi], hi = log2(8 (max D - min D)), keeping hi when the
  candidate fits, and returns the assignment at hi.
* App. B: the refit is a least-squares refit.  App. A: s and o become fp16
  ahead of the second Drift, whose assignment then targets exactly the levels
  the decoder reconstructs.

Readings (all arithmetic is fp64 with a fixed operation order, no fused
multiply-add; where floating point decides an integer both sides of a parity
test take the decision in the same precision)
-------------------------------------------------------------------------------
* Q1 D_im = e * e with t = s*m, u = o + t, e = x_i - u.
* Q2 hi is the integer ceil(log2(8 (max D - min D))) (exact through frexp);
  lambda runs on the grid 2**(U/512), U integer, so the 40-octave bracket is
  20480 units and all 12 midpoints are integers.
* Q3 the Lagrangian cost of (i, m) is D_im + lambda * r_m with
  r_m = R_m / 2**16 (exact); ties go to the smallest m.  The budget test uses
  the exact Q16 integer sum of R.
* Q4 if max D = min D every value takes the cheapest symbol (lowest index).
* Q5 if the assignment at the final hi still exceeds the budget (the initial
  bracket was too low), every value takes the nearest symbol among those of
  minimum cost.
* Q6 refit: S_m = sum m, S_mm = sum m^2 (integers); S_x = sum x,
  S_mx = sum m x as fold-in-halves fp64 trees (v[i] += v[i + len/2] until one
  element is left); den = n S_mm - S_m^2; s = (n S_mx - S_m S_x)/den;
  o = (S_x - s S_m)/n.  When den = 0, s is not finite or s <= 0 the min-max fit
  is kept.
* Q7 fp16 metadata: fp16(fp32(s)) and fp16(fp32(o)), both round-to-nearest-even.
"""

from __future__ import annotations

import numpy as np

from .tables import Tables, Q16, LAMBDA_STEPS

BISECT_STEPS = 12            # T in Alg. 1
BRACKET_OCTAVES = 40         # hi - lo in Alg. 1
BRACKET_UNITS = BRACKET_OCTAVES * LAMBDA_STEPS


def fold_sum(v: np.ndarray) -> np.ndarray:
    """Fold-in-halves fp64 tree sum over the last axis (length a power of 2)."""
    v = np.asarray(v, dtype=np.float64)
    while v.shape[-1] > 1:
        h = v.shape[-1] // 2
        v = v[..., :h] + v[..., h:]
    return v[..., 0]


def fit_minmax(x: np.ndarray, M: int):
    """Eq. (affine_token): s = (max - min)/(M - 1), o = min (fp64)."""
    mn = x.min(axis=-1)
    mx = x.max(axis=-1)
    return (mx - mn) / float(M - 1), mn


def distortion(x: np.ndarray, s: np.ndarray, o: np.ndarray, M: int) -> np.ndarray:
    """D[S, n, M] following reading Q1."""
    m = np.arange(M, dtype=np.float64)
    t = s[:, None] * m[None, :]
    u = o[:, None] + t
    e = x[:, :, None] - u[:, None, :]
    return e * e


def lam_of_units(U: np.ndarray, lam32: np.ndarray) -> np.ndarray:
    """lambda(U) = Lambda[U mod 512] * 2**floor(U / 512) (reading Q2)."""
    U = np.asarray(U, dtype=np.int64)
    base = lam32.astype(np.float64)[U & (LAMBDA_STEPS - 1)]
    return np.ldexp(base, (U >> 9).astype(np.int64))


def assign(D: np.ndarray, lam: np.ndarray, rate: np.ndarray) -> np.ndarray:
    """argmin_m D_im + lambda r_m per value, ties to the smallest m (Q3)."""
    pen = lam[:, None] * rate[None, :]              # [S, M], fp64 product
    J = D + pen[:, None, :]
    return np.argmin(J, axis=-1)


def drift(x: np.ndarray, s: np.ndarray, o: np.ndarray, tab: Tables,
          budget_q16: np.ndarray, trace: dict | None = None) -> np.ndarray:
    """Drift(x, s, o, r, B) of Alg. 1 for a batch of streams x[S, n].

    If `trace` is a dict it receives the bisection bracket per stream, in
    lambda-grid units: "U_hi0" / "U_lo0" (the initial hi and lo), "U_hi" (the
    final hi, whose assignment is returned unless reading Q5 or Q4 applies)
    and "flat" (reading Q4)."""
    S = x.shape[0]
    M = tab.M
    rate = tab.rate
    cost = tab.cost
    budget_q16 = np.broadcast_to(np.asarray(budget_q16, dtype=np.int64), (S,))
    D = distortion(x, s, o, M)
    Dmax = D.max(axis=(1, 2))
    Dmin = D.min(axis=(1, 2))
    flat = Dmax == Dmin
    delta = 8.0 * (Dmax - Dmin)
    mant, ex = np.frexp(np.where(flat, 1.0, delta))
    hi = np.where(mant == 0.5, ex - 1, ex).astype(np.int64)
    U_hi = hi * LAMBDA_STEPS
    U_lo = U_hi - BRACKET_UNITS
    if trace is not None:
        trace.update(U_hi0=U_hi.copy(), U_lo0=U_lo.copy(), flat=flat.copy())
    for _ in range(BISECT_STEPS):
        U_mid = (U_lo + U_hi) >> 1
        m = assign(D, lam_of_units(U_mid, tab.lam), rate)
        fits = cost[m].sum(axis=1) <= budget_q16
        U_hi = np.where(fits, U_mid, U_hi)
        U_lo = np.where(fits, U_lo, U_mid)
    if trace is not None:
        trace["U_hi"] = U_hi.copy()
    m = assign(D, lam_of_units(U_hi, tab.lam), rate)
    over = cost[m].sum(axis=1) > budget_q16
    if np.any(over):
        cheap = cost == cost.min()
        Dc = np.where(cheap[None, None, :], D, np.inf)
        m_cheap = np.argmin(Dc, axis=-1)
        m = np.where(over[:, None], m_cheap, m)
    if np.any(flat):
        m = np.where(flat[:, None], tab.cheapest, m)
    return m.astype(np.int64)


def refit(x: np.ndarray, m: np.ndarray, s0: np.ndarray, o0: np.ndarray):
    """Least-squares refit of (s, o) to the assignment (reading Q6), fp64."""
    n = x.shape[1]
    Sm = m.sum(axis=1)
    Smm = (m * m).sum(axis=1)
    Sx = fold_sum(x)
    Smx = fold_sum(m.astype(np.float64) * x)
    den_i = n * Smm - Sm * Sm
    den = den_i.astype(np.float64)
    Smf = Sm.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        s = (float(n) * Smx - Smf * Sx) / den
        o = (Sx - s * Smf) / float(n)
    bad = (den_i == 0) | ~np.isfinite(s) | (s <= 0)
    return np.where(bad, s0, s), np.where(bad, o0, o)


def to_fp16(v: np.ndarray) -> np.ndarray:
    """Reading Q7: fp16(fp32(v)), round to nearest even at both steps."""
    with np.errstate(over="ignore"):
        return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float16)


def first_pass(x: np.ndarray, tab: Tables):
    """Alg. 1 up to the fp16 metadata: returns (s16, o16) for streams x[S, n]."""
    s0, o0 = fit_minmax(x, tab.M)
    m1 = drift(x, s0, o0, tab, tab.budget_q16)
    s1, o1 = refit(x, m1, s0, o0)
    return to_fp16(s1), to_fp16(o1)


def final_drift(x: np.ndarray, s16: np.ndarray, o16: np.ndarray, tab: Tables,
                budget_q16) -> np.ndarray:
    """The second Drift of Alg. 1, on the fp16 grid."""
    return drift(x, s16.astype(np.float64), o16.astype(np.float64), tab, budget_q16)
