"""Pins for the oracle's FitMinMax / Drift / Refit (Alg. 1), CPU only."""

import itertools

import numpy as np
import pytest

from oracle import kv, quantize, tables


def _tab(M, C, n=128, alpha=1.4, p=12):
    return tables.build_tables(n, M, p, alpha, C)


@pytest.mark.parametrize("M,C", [(6, 36), (5, 32), (9, 48), (17, 64)])
def test_drift_respects_budget(M, C):
    t = _tab(M, C)
    rng = np.random.default_rng(M)
    x = rng.normal(size=(400, 128)) * rng.uniform(0.1, 10, size=(400, 1)) + rng.normal(size=(400, 1))
    s, o = quantize.fit_minmax(x, M)
    m = quantize.drift(x, s, o, t, t.budget_q16)
    assert np.all(t.cost[m].sum(axis=1) <= t.budget_q16)
    assert m.min() >= 0 and m.max() < M


def test_generous_budget_is_nearest_rounding():
    """With room for every symbol the Lagrangian optimum is textbook
    round-to-nearest on the grid (lambda -> lower end of the bracket)."""
    t = _tab(8, 400)
    rng = np.random.default_rng(5)
    x = rng.normal(size=(200, 128))
    s, o = quantize.fit_minmax(x, 8)
    m = quantize.drift(x, s, o, t, t.budget_q16)
    ref = np.clip(np.rint((x - o[:, None]) / s[:, None]), 0, 7)
    assert np.mean(m == ref) > 0.999  # half-way ties may differ
    lv = o[:, None, None] + s[:, None, None] * np.arange(8)
    dist = np.abs(x[:, :, None] - lv)
    assert np.all(dist[np.arange(200)[:, None], np.arange(128)[None, :], m] <= dist.min(axis=-1) + 1e-12)


def test_lagrangian_optimality_brute_force():
    """The drift result minimizes Eq. (drift) among all assignments whose cost
    does not exceed its own (exhaustive over M**n, n = 7, M = 4)."""
    n, M = 7, 4
    # a budget that binds: about 1.2 bits per symbol of payload
    t = tables.build_tables(n, M, 12, 1.4, 100)
    rng = np.random.default_rng(11)
    allm = np.array(list(itertools.product(range(M), repeat=n)))
    Rall = t.cost[allm].sum(axis=1)
    for trial in range(25):
        x = rng.normal(size=(1, n))
        s, o = quantize.fit_minmax(x, M)
        budget = int(n * t.cost.min() + rng.integers(0, 6 * 65536))
        m = quantize.drift(x, s, o, t, budget)[0]
        R = int(t.cost[m].sum())
        assert R <= budget
        lv = o[0] + s[0] * np.arange(M)
        Dall = ((x[0][None, :] - lv[allm]) ** 2).sum(axis=1)
        D = ((x[0] - lv[m]) ** 2).sum()
        better = (Rall <= R) & (Dall < D - 1e-12)
        assert not better.any(), trial


def test_cost_monotone_in_lambda():
    t = _tab(9, 48)
    rng = np.random.default_rng(2)
    x = rng.normal(size=(50, 128))
    s, o = quantize.fit_minmax(x, 9)
    D = quantize.distortion(x, s, o, 9)
    prev = None
    for U in range(-15000, 4000, 137):
        m = quantize.assign(D, quantize.lam_of_units(np.full(50, U), t.lam), t.rate)
        c = t.cost[m].sum(axis=1)
        if prev is not None:
            assert np.all(c <= prev)
        prev = c


def test_lambda_grid():
    lam = tables.lambda_table()
    U = np.array([0, 512, -512, 256, 513, -1])
    v = quantize.lam_of_units(U, lam)
    assert v[0] == 1.0 and v[1] == 2.0 and v[2] == 0.5
    assert v[3] == np.float64(np.float32(np.sqrt(2.0)))
    assert v[4] == 2.0 * np.float64(lam[1])
    assert v[5] == 0.5 * np.float64(lam[511])


def test_flat_stream_takes_cheapest_symbol():
    t = _tab(6, 36)
    x = np.full((3, 128), 0.75)
    s, o = quantize.fit_minmax(x, 6)
    m = quantize.drift(x, s, o, t, t.budget_q16)
    assert np.all(m == t.cheapest)
    s16, o16 = quantize.first_pass(x, t)
    assert np.all(s16 == 0) and np.all(o16 == np.float16(0.75))


def test_rate_minimal_fallback():
    """When the assignment at the top of the bracket still overflows, every
    value takes the nearest minimum-cost symbol (reading Q5)."""
    t = _tab(4, 64)
    # nearly uniform costs so that lambda = 8 (max D - min D) cannot force
    # the cheap symbols
    t.freq = np.array([1020, 1028, 1028, 1020], dtype=np.int64)
    t.cum = np.concatenate([[0], np.cumsum(t.freq)[:-1]])
    t.cost = tables.cost_q16(t.freq, 12)
    rng = np.random.default_rng(3)
    x = rng.normal(size=(20, 128))
    s, o = quantize.fit_minmax(x, 4)
    budget = 128 * int(t.cost.min())
    m = quantize.drift(x, s, o, t, budget)
    assert np.all(t.cost[m].sum(axis=1) <= budget)
    assert np.all((m == 1) | (m == 2))
    lv = o[:, None] + s[:, None] * np.array([1.0, 2.0])
    near = np.where(np.abs(x - lv[:, :1]) <= np.abs(x - lv[:, 1:]), 1, 2)
    assert np.array_equal(m, near)


def test_refit_is_least_squares():
    rng = np.random.default_rng(7)
    x = rng.normal(size=(30, 128)) * 3 + 1
    m = rng.integers(0, 8, size=(30, 128))
    s, o = quantize.refit(x, m, np.ones(30), np.zeros(30))
    for i in range(30):
        A = np.stack([np.ones(128), m[i].astype(float)], axis=1)
        (o_ref, s_ref), *_ = np.linalg.lstsq(A, x[i], rcond=None)
        if s_ref > 0:
            assert abs(s[i] - s_ref) < 1e-12 * max(1, abs(s_ref))
            assert abs(o[i] - o_ref) < 1e-12 * max(1, abs(o_ref))
        else:
            assert s[i] == 1 and o[i] == 0


def test_refit_degenerate_keeps_minmax():
    x = np.random.default_rng(0).normal(size=(2, 128))
    m = np.full((2, 128), 3)
    s, o = quantize.refit(x, m, np.array([0.5, 0.25]), np.array([-1.0, 2.0]))
    assert np.array_equal(s, [0.5, 0.25]) and np.array_equal(o, [-1.0, 2.0])


def test_fold_sum_order():
    v = np.array([1e16, 1.0, -1e16, 1.0])
    # (1e16 + -1e16) + (1 + 1) = 2 in fold-in-halves order
    assert quantize.fold_sum(v) == 2.0
    assert quantize.to_fp16(np.array([65504.0]))[0] == np.float16(65504)
    assert np.isinf(quantize.to_fp16(np.array([1e6]))[0])


def test_fp16_metadata_is_what_the_record_uses():
    """App. A: the final assignment is made against the fp16 grid."""
    t = _tab(6, 36)
    rng = np.random.default_rng(1)
    x = rng.normal(size=(64, 128)) * 7.3 + 0.1
    recs, syms, s16, o16, budgets = kv.encode_streams(x, t)
    m2 = quantize.final_drift(x, s16, o16, t, budgets)
    assert np.array_equal(m2, syms)


# ---- the bisection schedule of Alg. 1: hi = ceil(log2(8 (max D - min D))),
#      lo = hi - 40 octaves, T = 12 halvings, answer at the final hi

def _fits(D, U, t, budget):
    m = quantize.assign(D, quantize.lam_of_units(U, t.lam), t.rate)
    return t.cost[m].sum(axis=1) <= budget


def _schedule_violations(x, s, o, t, budget):
    """Streams whose Drift bracket contradicts Alg. 1's schedule."""
    tr = {}
    m = quantize.drift(x, s, o, t, budget, trace=tr)
    D = quantize.distortion(x, s, o, t.M)
    live = ~tr["flat"]
    delta = 8.0 * (D.max(axis=(1, 2)) - D.min(axis=(1, 2)))
    U_hi0, U_lo0, U_hi = tr["U_hi0"], tr["U_lo0"], tr["U_hi"]
    bad = np.zeros(x.shape[0], dtype=bool)
    # the initial hi is the integer ceiling of log2(8 dD): 2^(hi-1) < 8 dD <= 2^hi
    hi0 = U_hi0 // 512
    bad |= live & ((U_hi0 % 512 != 0) | ~(np.ldexp(1.0, hi0 - 1) < delta) | ~(delta <= np.ldexp(1.0, hi0)))
    # a 40-octave bracket on the 1/512-octave grid
    bad |= live & (U_hi0 - U_lo0 != 40 * 512)
    # twelve halvings of 20480 units leave brackets of 5 units: the final hi
    # lies on that grid, it fits, and one step below it does not (unless that
    # is the bracket's untested lower end)
    fits_hi = _fits(D, U_hi, t, budget)
    fits_below = _fits(D, U_hi - 5, t, budget)
    bad |= live & ((U_hi0 - U_hi) % 5 != 0)
    bad |= live & fits_hi & fits_below & (U_hi - 5 != U_lo0)
    # the result is the assignment at the final hi whenever that fits
    at_hi = quantize.assign(D, quantize.lam_of_units(U_hi, t.lam), t.rate)
    bad |= live & fits_hi & np.any(m != at_hi, axis=1)
    return bad, live & fits_hi


def _schedule_inputs():
    rng = np.random.default_rng(19)
    x = rng.normal(size=(300, 128)) * rng.uniform(0.05, 20, size=(300, 1)) + rng.normal(size=(300, 1))
    x[::7, :3] *= 9.0          # outliers, as rotated keys carry
    return x


@pytest.mark.parametrize("M,C", [(6, 36), (5, 32), (9, 48), (17, 64)])
def test_drift_bisection_schedule(M, C):
    """Both drifts of Alg. 1 follow its schedule exactly on every stream."""
    t = _tab(M, C)
    x = _schedule_inputs()
    s0, o0 = quantize.fit_minmax(x, M)
    bad, checked = _schedule_violations(x, s0, o0, t, t.budget_q16)
    assert not bad.any()
    assert checked.sum() > 250
    s16, o16 = quantize.first_pass(x, t)
    bad, checked = _schedule_violations(x, s16.astype(np.float64), o16.astype(np.float64), t, t.budget_q16)
    assert not bad.any()


@pytest.mark.parametrize("steps,octaves", [(11, 40), (13, 40), (12, 20), (12, 41)])
def test_drift_schedule_pin_catches_a_wrong_schedule(monkeypatch, steps, octaves):
    """Plants a wrong T or bracket in the oracle: the schedule pin fails."""
    monkeypatch.setattr(quantize, "BISECT_STEPS", steps)
    monkeypatch.setattr(quantize, "BRACKET_UNITS", octaves * 512)
    t = _tab(6, 36)
    x = _schedule_inputs()
    s0, o0 = quantize.fit_minmax(x, 6)
    bad, _ = _schedule_violations(x, s0, o0, t, t.budget_q16)
    assert bad.any()
