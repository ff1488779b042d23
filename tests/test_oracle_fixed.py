"""Pins of the oracle's fixed-width comparator (App. B; oracle/fixed.py), CPU.

* Sec. 3's INT2 example: 128 values with an fp16 scale and zero point in 2.25
  bits per value is exactly the 36-byte record, b = 2 bits, 4 levels.
* The bit layout, written out by hand for a few symbols.
* Nearest-level rounding equals the textbook clip(rint((x - o) / s)) away
  from ties, and reconstructs values on the grid exactly.
* App. B's direction: at matched storage D-Quant's reconstruction error is
  below the fixed-width one (N(0,1) streams, 36-byte records).
* App. B's level counts at the per-token operating point: charged the ideal
  log2 M bits, 335 / 235-byte records of 1024 values allow 6 key and 3 value
  levels; D-Quant's 8 / 6 levels reconstruct N(0,1) tokens with less error.
"""

import numpy as np

from oracle import fixed, kv, tables


def test_int2_is_the_36_byte_record():
    assert fixed.bits_per_symbol(128, 36) == 2
    assert 36 * 8 / 128 == 2.25                        # Sec. 3: INT2 + fp16 s, o per 128 values
    assert fixed.bits_per_symbol(128, 32) == 1
    assert fixed.bits_per_symbol(128, 48) == 2
    assert fixed.bits_per_symbol(128, 68) == 4


def test_bit_layout_by_hand():
    sym = np.zeros((1, 128), dtype=np.int64)
    sym[0, :5] = [1, 2, 3, 0, 3]
    rec = fixed.pack(sym, np.array([1.0], np.float16), np.array([-2.0], np.float16), 2, 36)
    assert rec.shape == (1, 36)
    assert list(rec[0, :4]) == [0x00, 0x3C, 0x00, 0xC0]          # fp16 1.0 and -2.0, little-endian
    assert rec[0, 4] == (1 | 2 << 2 | 3 << 4 | 0 << 6)
    assert rec[0, 5] == 3 and not rec[0, 6:].any()
    back, s, o = fixed.unpack(rec, 128, 2)
    assert np.array_equal(back, sym) and float(s[0]) == 1.0 and float(o[0]) == -2.0
    rng = np.random.default_rng(0)
    for b, C in ((1, 32), (2, 36), (3, 64), (4, 68)):
        sym = rng.integers(0, 1 << b, size=(7, 128))
        rec = fixed.pack(sym, np.ones(7, np.float16), np.zeros(7, np.float16), b, C)
        assert np.array_equal(fixed.unpack(rec, 128, b)[0], sym)


def test_nearest_is_rounding():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(50, 128))
    s = rng.uniform(0.2, 1.0, size=50)
    o = rng.uniform(-3, -1, size=50)
    m = fixed.nearest(x, s, o, 8)
    ref = np.clip(np.rint((x - o[:, None]) / s[:, None]), 0, 7)
    assert np.array_equal(m, ref.astype(np.int64))
    grid = o[:, None] + s[:, None] * rng.integers(0, 8, size=(50, 128))
    mg = fixed.nearest(grid, s, o, 8)
    assert np.allclose(o[:, None] + s[:, None] * mg, grid, rtol=0, atol=1e-12)


def test_entropy_coding_beats_fixed_width_at_matched_storage():
    rng = np.random.default_rng(2)
    x = rng.normal(size=(1000, 128))
    m, s16, o16 = fixed.quantize_streams(x, 4)
    xf = s16.astype(np.float64)[:, None] * m + o16.astype(np.float64)[:, None]
    t = tables.build_tables(128, 6, 12, 1.4, 36)
    _, sym, ds, do, _ = kv.encode_streams(x, t)
    xd = ds.astype(np.float64)[:, None] * sym + do.astype(np.float64)[:, None]
    e_fixed = ((x - xf) ** 2).sum() / (x ** 2).sum()
    e_dq = ((x - xd) ** 2).sum() / (x ** 2).sum()
    assert e_dq < 0.9 * e_fixed, (e_dq, e_fixed)
    # the fixed-width quantizer keeps the least-squares refit: no worse than min-max
    s0, o0 = (x.max(1) - x.min(1)) / 3, x.min(1)
    m0 = fixed.nearest(x, s0, o0, 4)
    e0 = ((x - (s0[:, None] * m0 + o0[:, None])) ** 2).sum() / (x ** 2).sum()
    assert e_fixed < e0


def test_ideal_levels_at_the_paper_operating_points():
    assert fixed.ideal_levels(1024, 335) == 6          # App. B: 6 key levels
    assert fixed.ideal_levels(1024, 235) == 3          # App. B: 3 value levels
    assert fixed.ideal_levels(128, 36) == 4            # INT2, the stored format at 36 bytes
    assert fixed.ideal_levels(128, 36) == 1 << fixed.bits_per_symbol(128, 36)
    assert 1024 * np.log2(6) <= 8 * 331 < 1024 * np.log2(7)
    assert 1024 * np.log2(3) <= 8 * 231 < 1024 * np.log2(4)


def test_entropy_coding_beats_fixed_width_at_the_per_token_point():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(200, 1024))
    for C, M_dq in ((335, 8), (235, 6)):
        M_fx = fixed.ideal_levels(1024, C)
        m, s16, o16 = fixed.quantize_streams(x, M_fx)
        xf = s16.astype(np.float64)[:, None] * m + o16.astype(np.float64)[:, None]
        t = tables.build_tables(1024, M_dq, 8, 1.4, C)
        _, sym, ds, do, _ = kv.encode_streams(x, t)
        xd = ds.astype(np.float64)[:, None] * sym + do.astype(np.float64)[:, None]
        e_fixed = ((x - xf) ** 2).sum() / (x ** 2).sum()
        e_dq = ((x - xd) ** 2).sum() / (x ** 2).sum()
        assert e_dq < 0.75 * e_fixed, (C, e_dq, e_fixed)
