"""Pins for the oracle's rANS coder and record layout (CPU only)."""

import numpy as np
import pytest

from oracle import rans, tables


def _uniform_tables(M, p, C, n=128):
    t = tables.build_tables(n, M, p, 1.0, C)
    t.freq = np.full(M, (1 << p) // M, dtype=np.int64)
    t.cum = np.arange(M, dtype=np.int64) * ((1 << p) // M)
    t.cost = tables.cost_q16(t.freq, p)
    t.sym_of_z = np.repeat(np.arange(M), t.freq)
    return t


@pytest.mark.parametrize("M,p", [(6, 12), (16, 12), (5, 8), (64, 12), (9, 10)])
def test_round_trip_random(M, p):
    t = tables.build_tables(128, M, p, 1.4, 64)
    rng = np.random.default_rng(M)
    probs = t.freq / t.freq.sum()
    sym = rng.choice(M, size=(300, 128), p=probs)
    state, body, length = rans.encode(sym, t)
    assert np.all((state >= rans.RANS_L) & (state < 256 * rans.RANS_L))
    C = 8 + int(length.max())
    recs = rans.pack(np.ones(300, np.float16), np.zeros(300, np.float16), state, body, length, C)
    out, x, ptr = rans.decode(recs, t, 128)
    assert np.array_equal(out, sym)
    assert np.all(x == rans.RANS_L)
    assert np.array_equal(ptr, 8 + length)
    # emitted bits track the ideal cost: 8E within (sum r - 8, sum r + 1]
    ideal = t.rate[sym].sum(axis=1)
    assert np.all(8 * length > ideal - 8 - 1e-9)
    assert np.all(8 * length <= ideal + 1.0)


@pytest.mark.parametrize("which", ["rarest", "commonest", "alternate"])
def test_round_trip_adversarial(which):
    t = tables.build_tables(128, 16, 12, 1.4, 64)
    if which == "rarest":
        sym = np.zeros((2, 128), dtype=np.int64)
        sym[1] = 15
    elif which == "commonest":
        sym = np.full((2, 128), 7, dtype=np.int64)
        sym[1] = 8
    else:
        sym = np.tile(np.array([0, 15, 7, 8]), (2, 32))
    state, body, length = rans.encode(sym, t)
    recs = rans.pack(np.ones(2, np.float16), np.zeros(2, np.float16), state, body, length, 8 + int(length.max()))
    out, x, _ = rans.decode(recs, t, 128)
    assert np.array_equal(out, sym) and np.all(x == rans.RANS_L)


def test_uniform_alphabet_packs_exact_bits():
    """With a uniform table rANS is plain bit packing: k bits per symbol, so
    a stream of n symbols emits exactly floor(k n / 8) bytes."""
    for M, k in ((4, 2), (16, 4), (2, 1)):
        t = _uniform_tables(M, 12, 64)
        rng = np.random.default_rng(k)
        sym = rng.integers(0, M, size=(50, 128))
        _, _, length = rans.encode(sym, t)
        assert np.all(length == (k * 128) // 8)


def test_decoder_reads_at_most_two_bytes_per_symbol():
    # reading R1: x in [2^21, 2^29) and f >= 1 give x' >= 2^9 after a step
    t = tables.build_tables(128, 64, 12, 7.8, 64)
    sym = np.zeros((1, 128), dtype=np.int64)       # rarest symbol, f = 1
    _, _, length = rans.encode(sym, t)
    assert length[0] <= 2 * 128


def test_record_layout():
    t = tables.build_tables(128, 6, 12, 1.4, 36)
    sym = np.full((1, 128), 2, dtype=np.int64)
    state, body, length = rans.encode(sym, t)
    s16 = np.array([1.5], np.float16)
    o16 = np.array([-2.25], np.float16)
    rec = rans.pack(s16, o16, state, body, length, 36)
    assert rec.shape == (1, 36)
    assert int(rec[0, 0]) | (int(rec[0, 1]) << 8) == int(s16.view(np.uint16)[0])
    assert int(rec[0, 2]) | (int(rec[0, 3]) << 8) == int(o16.view(np.uint16)[0])
    st = int(rec[0, 4]) | int(rec[0, 5]) << 8 | int(rec[0, 6]) << 16 | int(rec[0, 7]) << 24
    assert st == int(state[0])
    k = int(length[0])
    assert np.all(rec[0, 8 + k:] == 0)
    s, o = rans.unpack_header(rec)
    assert s[0] == s16[0] and o[0] == o16[0]


def test_corrupted_record_is_detected():
    t = tables.build_tables(128, 6, 12, 1.4, 36)
    rng = np.random.default_rng(9)
    sym = rng.choice(6, size=(64, 128), p=t.freq / 4096)
    state, body, length = rans.encode(sym, t)
    recs = rans.pack(np.ones(64, np.float16), np.zeros(64, np.float16), state, body, length, 8 + int(length.max()))
    bad = recs.copy()
    bad[:, 5] ^= 0x5A
    _, x, _ = rans.decode(bad, t, 128)
    assert np.mean(x != rans.RANS_L) > 0.9


def test_all_zero_record_terminates():
    t = tables.build_tables(128, 6, 12, 1.4, 36)
    _, x, ptr = rans.decode(np.zeros((3, 36), np.uint8), t, 128)
    assert np.all(x != rans.RANS_L) and np.all(ptr <= 36)
