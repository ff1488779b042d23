"""Pins for the oracle's fp64 attention (CPU only)."""

import numpy as np
import pytest
import scipy.linalg
import scipy.special

from oracle import attention


def _random_cache(rng, B, Hkv, T, d, M, window):
    k_sym = rng.integers(0, M, size=(B, Hkv, T, d))
    v_sym = rng.integers(0, M, size=(B, Hkv, T, d))
    k_s = rng.uniform(0.1, 2, size=(B, Hkv, T)).astype(np.float16)
    k_o = rng.normal(size=(B, Hkv, T)).astype(np.float16)
    v_s = rng.uniform(0.1, 2, size=(B, Hkv, T)).astype(np.float16)
    v_o = rng.normal(size=(B, Hkv, T)).astype(np.float16)
    mean = rng.normal(size=(B, Hkv, -(-T // window), d))
    return k_sym, k_s, k_o, mean, v_sym, v_s, v_o


def test_brute_force_tiny():
    """B = 1, Hq = 2, Hkv = 1, d = 8, T = 3 against softmax(q K^T / sqrt d) V
    built by hand from an explicit Hadamard matrix."""
    rng = np.random.default_rng(0)
    d, T, M, W = 8, 3, 5, 4
    k_sym, k_s, k_o, mean, v_sym, v_s, v_o = _random_cache(rng, 1, 1, T, d, M, W)
    q = rng.normal(size=(1, 2, d))
    H = scipy.linalg.hadamard(d).astype(float)
    k_rot = k_s[0, 0].astype(float)[:, None] * k_sym[0, 0] + k_o[0, 0].astype(float)[:, None] + mean[0, 0, 0]
    v_rot = v_s[0, 0].astype(float)[:, None] * v_sym[0, 0] + v_o[0, 0].astype(float)[:, None]
    K = np.linalg.solve(H, k_rot.T).T      # undo the rotation by solving, not by H/d
    V = np.linalg.solve(H, v_rot.T).T
    ref = scipy.special.softmax(q[0] @ K.T / np.sqrt(d), axis=-1) @ V
    out = attention.attention_folded(q, k_sym, k_s, k_o, mean, v_sym, v_s, v_o, [T], 2, 1 / np.sqrt(d), window=W)
    assert np.max(np.abs(out[0] - ref)) < 1e-12
    krot = attention.dequantize(k_sym, k_s, k_o, mean, window=W)
    vrot = attention.dequantize(v_sym, v_s, v_o)
    out2 = attention.attention_direct(q, krot, vrot, [T], 2, 1 / np.sqrt(d))
    assert np.max(np.abs(out2[0] - ref)) < 1e-12


@pytest.mark.parametrize("G", [1, 4, 8])
def test_folded_equals_direct(G):
    """Eq. (fold-key) and Eq. (fold-value) are identities of the dequantized
    attention."""
    rng = np.random.default_rng(G)
    B, Hkv, T, d, M, W = 2, 2, 256, 32, 9, 128
    k_sym, k_s, k_o, mean, v_sym, v_s, v_o = _random_cache(rng, B, Hkv, T, d, M, W)
    q = rng.normal(size=(B, Hkv * G, d)) * 3
    lens = [256, 130]
    krot = attention.dequantize(k_sym, k_s, k_o, mean, window=W)
    vrot = attention.dequantize(v_sym, v_s, v_o)
    a = attention.attention_direct(q, krot, vrot, lens, G, 0.1)
    b = attention.attention_folded(q, k_sym, k_s, k_o, mean, v_sym, v_s, v_o, lens, G, 0.1, window=W)
    assert np.max(np.abs(a - b)) < 1e-11 * np.max(np.abs(a))


def test_gqa_mapping_and_lengths():
    rng = np.random.default_rng(4)
    B, Hkv, T, d, M = 1, 2, 8, 8, 4
    k_sym, k_s, k_o, _, v_sym, v_s, v_o = _random_cache(rng, B, Hkv, T, d, M, 8)
    q = rng.normal(size=(B, 4, d))
    out = attention.attention_folded(q, k_sym, k_s, k_o, None, v_sym, v_s, v_o, [5], 2, 0.3, window=8)
    # heads 2, 3 use kv head 1: recompute with kv head 1 copied into slot 0
    k2 = [a.copy() for a in (k_sym, k_s, k_o, v_sym, v_s, v_o)]
    for a in k2:
        a[:, 0] = a[:, 1]
    out2 = attention.attention_folded(q[:, 2:], k2[0], k2[1], k2[2], None, k2[3], k2[4], k2[5], [5], 2, 0.3, window=8)
    assert np.max(np.abs(out[:, 2:] - out2)) < 1e-13
    # tokens past the length do not matter
    k3 = k_sym.copy()
    k3[..., 5:, :] = 0
    out3 = attention.attention_folded(q, k3, k_s, k_o, None, v_sym, v_s, v_o, [5], 2, 0.3, window=8)
    assert np.array_equal(out, out3)


# ---------------------------------------------------------------- residual window

def test_residual_only_is_plain_attention():
    """With no compressed tokens the residual window is plain softmax attention
    over the raw tokens (scipy's softmax as the reference)."""
    rng = np.random.default_rng(11)
    B, Hkv, G, R, d = 2, 2, 3, 17, 16
    q = rng.normal(size=(B, Hkv * G, d))
    rk = rng.normal(size=(B, Hkv, R, d))
    rv = rng.normal(size=(B, Hkv, R, d))
    lens = [R, 5]
    empty = np.zeros((B, Hkv, 0, d))
    out = attention.attention_with_residual(q, empty, empty, [0, 0], rk, rv, lens, G, 0.3)
    for b in range(B):
        for i in range(Hkv * G):
            h = i // G
            ref = scipy.special.softmax(0.3 * rk[b, h, :lens[b]] @ q[b, i]) @ rv[b, h, :lens[b]]
            assert np.max(np.abs(out[b, i] - ref)) < 1e-13


def test_residual_empty_equals_compressed_attention():
    rng = np.random.default_rng(12)
    B, Hkv, G, T, d, M, W = 2, 1, 4, 200, 32, 6, 128
    k_sym, k_s, k_o, mean, v_sym, v_s, v_o = _random_cache(rng, B, Hkv, T, d, M, W)
    q = rng.normal(size=(B, Hkv * G, d))
    krot = attention.dequantize(k_sym, k_s, k_o, mean, window=W)
    vrot = attention.dequantize(v_sym, v_s, v_o)
    rk = rng.normal(size=(B, Hkv, 8, d))
    a = attention.attention_with_residual(q, krot, vrot, [T, 77], rk, rk, [0, 0], G, 0.2)
    b = attention.attention_direct(q, krot, vrot, [T, 77], G, 0.2)
    assert np.max(np.abs(a - b)) < 1e-13 * np.max(np.abs(b))


def test_residual_split_point_is_invisible():
    """Raw tokens stored as exact rotated reconstructions (k_rot = k H) give
    the same result whichever of them are called compressed: the basis change
    and the union of the two sets are both right."""
    rng = np.random.default_rng(13)
    B, Hkv, G, N, d = 1, 2, 2, 40, 16
    H = scipy.linalg.hadamard(d).astype(float)
    k = rng.normal(size=(B, Hkv, N, d))
    v = rng.normal(size=(B, Hkv, N, d))
    q = rng.normal(size=(B, Hkv * G, d))
    full = attention.attention_with_residual(q, np.zeros((B, Hkv, 0, d)), np.zeros((B, Hkv, 0, d)), [0],
                                             k, v, [N], G, 0.25)
    for T in (1, 13, 39, N):
        out = attention.attention_with_residual(q, k[:, :, :T] @ H, v[:, :, :T] @ H, [T],
                                                k[:, :, T:], v[:, :, T:], [N - T], G, 0.25)
        assert np.max(np.abs(out - full)) < 1e-12


def test_residual_order_and_empty_sequence():
    rng = np.random.default_rng(14)
    B, Hkv, G, R, d = 2, 1, 2, 9, 8
    q = rng.normal(size=(B, Hkv * G, d))
    rk = rng.normal(size=(B, Hkv, R, d))
    rv = rng.normal(size=(B, Hkv, R, d))
    e = np.zeros((B, Hkv, 0, d))
    perm = rng.permutation(R)
    a = attention.attention_with_residual(q, e, e, [0, 0], rk, rv, [R, 0], G, 0.5)
    b = attention.attention_with_residual(q, e, e, [0, 0], rk[:, :, perm], rv[:, :, perm], [R, 0], G, 0.5)
    assert np.max(np.abs(a - b)) < 1e-13
    assert np.all(a[1] == 0.0)        # a sequence with no tokens gives 0


def test_empty_sequence_gives_zero():
    """Reading A3: a sequence with no tokens gives 0, in every form."""
    rng = np.random.default_rng(15)
    B, Hkv, T, d, M, W = 2, 1, 128, 16, 5, 128
    k_sym, k_s, k_o, mean, v_sym, v_s, v_o = _random_cache(rng, B, Hkv, T, d, M, W)
    q = rng.normal(size=(B, 2, d))
    krot = attention.dequantize(k_sym, k_s, k_o, mean, window=W)
    vrot = attention.dequantize(v_sym, v_s, v_o)
    a = attention.attention_direct(q, krot, vrot, [T, 0], 2, 0.3)
    b = attention.attention_folded(q, k_sym, k_s, k_o, mean, v_sym, v_s, v_o, [T, 0], 2, 0.3, window=W)
    assert np.all(a[1] == 0.0) and np.all(b[1] == 0.0)
    assert np.max(np.abs(a[0] - b[0])) < 1e-12 * np.max(np.abs(a[0]))
