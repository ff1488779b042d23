"""Pins for the oracle's entropy model and budget arithmetic (CPU only)."""

import math

import mpmath
import numpy as np
import pytest
import scipy.stats

from conftest import read_golden
from oracle import tables


def test_expected_max_closed_forms():
    # E[max of 2 normals] = 1/sqrt(pi), E[max of 3] = 3/(2 sqrt(pi))
    assert abs(tables.expected_max_normal(2) - 1 / math.sqrt(math.pi)) < 1e-13
    assert abs(tables.expected_max_normal(3) - 1.5 / math.sqrt(math.pi)) < 1e-13
    assert tables.expected_max_normal(1) == 0.0


@pytest.mark.parametrize("n", [16, 128, 1024])
def test_expected_max_independent_quadrature(n):
    mpmath.mp.dps = 30
    f = lambda x: x * n * mpmath.npdf(x) * mpmath.ncdf(x) ** (n - 1)  # noqa: E731
    ref = float(mpmath.quad(f, [-mpmath.inf, -4, 0, 2, 4, 8, mpmath.inf]))
    assert abs(tables.expected_max_normal(n) - ref) < 1e-11


def test_expected_max_monte_carlo():
    rng = np.random.default_rng(0)
    mx = rng.normal(size=(20000, 128)).max(axis=1)
    se = mx.std() / math.sqrt(mx.size)
    assert abs(mx.mean() - tables.expected_max_normal(128)) < 4 * se


@pytest.mark.parametrize("M", [2, 3, 5, 6, 8, 11, 16, 17, 32, 64])
def test_level_probabilities(M):
    q = tables.level_probabilities(128, M)
    assert abs(q.sum() - 1.0) < 1e-14
    assert np.all(q > 0)
    assert np.array_equal(q, q[::-1])
    # same masses through a different CDF routine
    a = tables.expected_max_normal(128)
    edges = np.concatenate([[-np.inf], a * ((2 * np.arange(1, M) - 1) / (M - 1) - 1), [np.inf]])
    ref = np.diff(scipy.stats.norm.cdf(edges))
    assert np.max(np.abs(q - ref)) < 1e-14


def test_level_probabilities_match_sampled_grid():
    # Quantize N(0,1) values on the grid [-a_n, a_n]: the plug-in model of
    # reading T1 is close to what a sample actually produces.
    rng = np.random.default_rng(1)
    x = rng.normal(size=(4000, 128))
    M = 8
    a = tables.expected_max_normal(128)
    m = np.clip(np.rint((x + a) / (2 * a) * (M - 1)), 0, M - 1).astype(int)
    freq = np.bincount(m.ravel(), minlength=M) / m.size
    q = tables.level_probabilities(128, M)
    assert np.max(np.abs(freq - q)) < 0.004


@pytest.mark.parametrize("M,p,alpha", [(6, 12, 1.4), (16, 12, 1.4), (16, 12, 5.6), (9, 12, 1.4),
                                       (17, 12, 1.4), (64, 12, 7.8), (5, 8, 1.4), (8, 10, 1.0),
                                       (32, 12, 7.6), (16, 12, 8.6), (64, 8, 1.4)])
def test_frequencies(M, p, alpha):
    qs = tables.sharpen(tables.level_probabilities(128, M), alpha)
    f = tables.quantize_frequencies(qs, p)
    assert f.sum() == 1 << p
    assert f.min() >= 1
    assert np.array_equal(f, f[::-1])
    # apportionment never moves a symbol by more than one unit beyond clamping
    g = qs * (1 << p)
    assert np.all(f <= np.maximum(1, np.floor(g)) + 2)
    assert np.all(f >= np.minimum(np.floor(g), f) - 2)


def test_sharpening_exponent():
    q = tables.level_probabilities(128, 6)
    s = tables.sharpen(q, 1.4)
    assert abs(s.sum() - 1) < 1e-15
    ratio = (s[2] / s[0]) / (q[2] / q[0]) ** 1.4
    assert abs(ratio - 1) < 1e-12
    assert s[2] > q[2]  # sharpening moves mass to the centre


WORKLOAD_TABLES = [(128, 6, 12, 1.4, 36), (128, 5, 12, 1.4, 32), (128, 9, 12, 1.4, 48),
                   (128, 17, 12, 1.4, 64), (128, 16, 12, 5.6, 36), (128, 16, 12, 8.6, 32),
                   (128, 32, 12, 7.6, 48), (128, 64, 12, 7.8, 64), (1024, 6, 12, 1.4, 235),
                   (1024, 8, 12, 1.4, 335)]


@pytest.mark.parametrize("n,M,p,alpha,C", WORKLOAD_TABLES)
def test_rounding_margins(n, M, p, alpha, C):
    """No rounding decision of the table build sits within 1e-9 of a tie, so a
    second implementation with a slightly different libm produces the same
    integers."""
    qs = tables.sharpen(tables.level_probabilities(n, M), alpha)
    g = qs[: M // 2] * (1 << p)
    frac = g - np.floor(g)
    assert np.all(np.minimum(frac, 1 - frac) > 1e-9)
    fr = np.sort(frac)
    assert np.all(np.diff(fr) > 1e-9)
    if M % 2:
        tot = g.sum() + 0.5
        assert abs(tot - round(tot)) > 1e-9
    t = tables.build_tables(n, M, p, alpha, C)
    r = (p - np.log2(t.freq.astype(np.float64))) * tables.Q16
    assert np.all(np.abs(r - np.floor(r) - 0.5) > 1e-6)
    lam = np.exp2(np.arange(512) / 512.0)
    # distance to the fp32 rounding boundary, relative
    f32 = lam.astype(np.float32).astype(np.float64)
    ulp = np.spacing(lam.astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(np.abs(lam - f32) - ulp / 2) / lam > 1e-14)


def test_costs_and_lut():
    t = tables.build_tables(128, 6, 12, 1.4, 36)
    ideal = -np.log2(t.freq / 4096.0)
    assert np.max(np.abs(t.rate - ideal)) <= 2.0 ** -17
    assert t.cum[0] == 0 and np.array_equal(np.diff(t.cum), t.freq[:-1])
    z = np.arange(4096)
    m = t.sym_of_z
    assert np.all(t.cum[m] <= z) and np.all(z < t.cum[m] + t.freq[m])
    assert t.cheapest == int(np.argmax(t.freq))


def test_lambda_table():
    lam = tables.lambda_table()
    assert lam.dtype == np.float32 and lam.shape == (512,)
    assert lam[0] == 1.0
    assert lam[256] == np.float32(math.sqrt(2.0))
    assert np.all(np.diff(lam) > 0) and lam[-1] < 2.0


def test_budget_arithmetic():
    # 36-byte record: 4 B metadata + 4 B state + 28 B of renorm bytes = 224 bits
    assert tables.record_budget_q16(36) == 224 << 16
    assert tables.record_bytes_for(2.26, 128) == 36
    assert tables.record_bytes_for(2.25, 128) == 36
    assert tables.record_bytes_for(2.0, 128) == 32
    assert tables.record_bytes_for(3.0, 128) == 48
    assert tables.record_bytes_for(4.0, 128) == 64


def test_storage_figures_of_the_paper():
    """Reading T4 reproduces the paper's bits-per-value figures."""
    rows = {r[0]: r for r in read_golden("storage.txt")}
    # INT2 + fp16 scale and zero point per 128 values
    g, _, bpv = int(rows["int2_group128"][1]), 0, float(rows["int2_group128"][3])
    assert abs((2 * g + 32) / g - bpv) < 1e-12
    # key: 331 B container + 4 B fp16 s,o + INT8 mean over 128 tokens (1024 B / 128 tokens)
    n, C, bpv = int(rows["key_container"][1]), int(rows["key_container"][2]), float(rows["key_container"][3])
    key = (8 * (C + 4) + 8 * n / 128) / n
    assert abs(key - bpv) < 0.005
    n, C, bpv = int(rows["value_container"][1]), int(rows["value_container"][2]), float(rows["value_container"][3])
    val = 8 * (C + 4) / n
    assert abs(val - bpv) < 0.005
    assert abs((key + val) / 2 - float(rows["average"][3])) < 0.005


def test_table2_feasibility_boundary():
    """Tab. 2: with 1024-value groups, the 231 B value container admits
    M <= 11 and rejects M = 12, 14; the 331 B key container admits every M in
    the table.  Reproduced with alpha = 1.4 and p = 12 (at alpha = 1.0 M = 11
    would not fit, so the boundary also pins the sharpening)."""
    for row in read_golden("table2_levels.txt"):
        M = int(row[0])
        v_ok = row[2] != "--"
        k_ok = row[1] != "--"
        assert tables.build_tables(1024, M, 12, 1.4, 231 + 4).feasible == v_ok, M
        assert tables.build_tables(1024, M, 12, 1.4, 331 + 4).feasible == k_ok, M
    assert not tables.build_tables(1024, 11, 12, 1.0, 235).feasible
