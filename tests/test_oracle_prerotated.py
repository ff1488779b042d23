"""Pins of the oracle's prerotated reading (Sec. 4.2: the value rotation can
be folded into the projection weights offline; readings V0 and A4), CPU only.

* Coding a tensor that arrives already rotated, with rotate_on=False, gives
  exactly the records of the online-rotation path on the unrotated tensor:
  ternary inputs make H x integer-valued (|H x| <= 128), so the pre-rotated
  input is exact in bf16 and the two paths see the same stream.
* With keys given as H k and the query as H q / d, the logits are those of
  the online path (H^T H = d I), so the outputs agree; with values given as
  H v the output comes back as H times the online output.
* Folded = direct, and both against a textbook softmax over the dequantized
  keys and values taken as they are (no basis change), on tiny inputs.
"""

import numpy as np
import pytest

import dq_workloads as wlmod
from oracle import attention, hadamard, kmean, kv, tables

D = 128


def _bf16(x64):
    """fp64 values that bf16 holds exactly -> bf16 bit patterns."""
    x32 = x64.astype(np.float32)
    bits = (x32.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal((bits.astype(np.uint32) << 16).view(np.float32), x32), "not exact in bf16"
    return bits


def _tabs():
    return tables.build_tables(D, 6, 12, 1.4, 36), tables.build_tables(D, 6, 12, 1.4, 36)


@pytest.mark.parametrize("seed", [0, 1])
def test_prerotated_records_equal_online_rotation(seed):
    tk, tv = _tabs()
    k = wlmod.bf16_bits(wlmod.make_ternary(seed, 1, 256, 2))
    v = wlmod.bf16_bits(wlmod.make_ternary(seed + 7, 1, 256, 2))
    hk = _bf16(hadamard.fwht(kv.bf16_to_f64(k)))
    hv = _bf16(hadamard.fwht(kv.bf16_to_f64(v)))
    r_on, mq_on, ms_on, s_on = kv.encode_keys(k, tk)
    r_pre, mq_pre, ms_pre, s_pre = kv.encode_keys(hk, tk, rotate_on=False)
    assert np.array_equal(r_on, r_pre) and np.array_equal(mq_on, mq_pre)
    assert np.array_equal(ms_on.view(np.uint16), ms_pre.view(np.uint16)) and np.array_equal(s_on, s_pre)
    rv_on, _ = kv.encode_values(v, tv)
    rv_pre, _ = kv.encode_values(hv, tv, rotate_on=False)
    assert np.array_equal(rv_on, rv_pre)
    # and not by accident: coding the rotated tensor with the rotation again differs
    assert not np.array_equal(kv.encode_values(hv, tv)[0], rv_on)


def test_prerotated_tokenwise_records_equal_online_rotation():
    tk = tables.build_tables(2 * D, 8, 8, 1.4, 88)
    k = wlmod.bf16_bits(wlmod.make_ternary(3, 1, 128, 2))
    hk = _bf16(hadamard.fwht(kv.bf16_to_f64(k)))
    a = kv.encode_keys_tokenwise(k, tk)
    b = kv.encode_keys_tokenwise(hk, tk, rotate_on=False)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))


def _decoded(tk, tv, k, v, rotate_on):
    krec, mq, ms, ksym = kv.encode_keys(k, tk, rotate_on=rotate_on)
    vrec, vsym = kv.encode_values(v, tv, rotate_on=rotate_on)
    _, ks, ko, _ = kv.decode_records(krec, tk, D)
    _, vs, vo, _ = kv.decode_records(vrec, tv, D)
    return ksym, ks, ko, kmean.dequantize_mean(mq, ms), vsym, vs, vo


def test_prerotated_attention_matches_online_path():
    tk, tv = _tabs()
    B, T, H, G = 2, 384, 2, 4
    k = wlmod.bf16_bits(wlmod.make_ternary(11, B, T, H))
    v = wlmod.bf16_bits(wlmod.make_ternary(12, B, T, H))
    q = kv.bf16_to_f64(wlmod.bf16_bits(wlmod.make_ternary(13, B, H * G, 1)[:, :, 0]))   # [B, Hq, d]
    lens = [T, 200]
    on = _decoded(tk, tv, k, v, True)
    out_on = attention.attention_folded(q, *on[:4], *on[4:], lens, G, 1 / np.sqrt(D))
    hk = _bf16(hadamard.fwht(kv.bf16_to_f64(k)))
    hv = _bf16(hadamard.fwht(kv.bf16_to_f64(v)))
    pre = _decoded(tk, tv, hk, hv, False)
    hq = hadamard.fwht(q) / D
    out_pre = attention.attention_folded(hq, *pre[:4], *pre[4:], lens, G, 1 / np.sqrt(D),
                                         rotate_k=False, rotate_v=False)
    # values given as H v: the output is H times the online output
    assert np.allclose(out_pre, hadamard.fwht(out_on), rtol=0, atol=1e-11 * np.abs(out_pre).max())
    # keys alone prerotated: the same output as the online path
    pre_k = _decoded(tk, tv, hk, v, False)
    pre_k = (pre_k[0], pre_k[1], pre_k[2], pre_k[3]) + on[4:]
    out_k = attention.attention_folded(hq, *pre_k[:4], *pre_k[4:], lens, G, 1 / np.sqrt(D), rotate_k=False)
    assert np.allclose(out_k, out_on, rtol=0, atol=1e-11 * np.abs(out_on).max())


def test_prerotated_folded_equals_direct_and_textbook():
    rng = np.random.default_rng(5)
    B, T, H, G, d = 1, 3, 1, 2, 8
    q = rng.normal(size=(B, H * G, d))
    ksym = rng.integers(0, 6, size=(B, H, T, d))
    vsym = rng.integers(0, 6, size=(B, H, T, d))
    ks, ko = rng.uniform(0.1, 1, size=(B, H, T)), rng.normal(size=(B, H, T))
    vs, vo = rng.uniform(0.1, 1, size=(B, H, T)), rng.normal(size=(B, H, T))
    k_hat = ks[..., None] * ksym + ko[..., None]
    v_hat = vs[..., None] * vsym + vo[..., None]
    scale = 0.3
    folded = attention.attention_folded(q, ksym, ks, ko, None, vsym, vs, vo, [T], G, scale, window=4,
                                        rotate_k=False, rotate_v=False)
    direct = attention.attention_direct(q, k_hat, v_hat, [T], G, scale, rotate_k=False, rotate_v=False)
    assert np.allclose(folded, direct, rtol=0, atol=1e-12)
    # textbook softmax(q k^T scale) v over the reconstructions as given
    for i in range(H * G):
        s = np.array([scale * float(np.dot(q[0, i], k_hat[0, 0, t])) for t in range(T)])
        a = np.exp(s - s.max())
        a = a / a.sum()
        ref = sum(a[t] * v_hat[0, 0, t] for t in range(T))
        assert np.allclose(folded[0, i], ref, rtol=0, atol=1e-12)
