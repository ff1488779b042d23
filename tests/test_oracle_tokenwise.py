"""Pins of the oracle's per-token streams (one stream of H d values per token,
spanning every KV head: Sec. 4.1, Sec. 4.5 "Decoding", Sec. 5.1), CPU only.

* With one KV head a token stream is the per-head stream: records, means and
  symbols equal the per-head encoder's, which the other oracle tests pin.
* Head order and the shared (s, o): the decoded token streams, split back into
  heads, reconstruct every head of the input; a transposed or shuffled head
  order, or a per-head affine, would not.
* Tab. 2 at the default operating point (331 B / 231 B containers with 8 / 6
  levels): N(0, 1) tokens give the paper's key and value NMSE within 15 %.
* The folded attention over token streams equals the textbook attention over
  their reconstruction.
"""

import numpy as np
import pytest

import dq_workloads as wlmod
from oracle import attention, hadamard, kmean, kv, tables


def _tabs():
    wl = wlmod.workload("b1_t4k_tok")
    tk = tables.build_tables(1024, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    tv = tables.build_tables(1024, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    return wl, tk, tv


def test_one_head_token_streams_are_head_streams():
    wl = wlmod.workload("b1_t4k")
    t = tables.build_tables(128, wl.k.levels, 12, wl.k.alpha, wl.k.record_bytes)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 3, batch=2, context=256))[:, :, 2:3]     # one KV head
    v = wlmod.bf16_bits(wlmod.make_v(wl, 3, batch=2, context=256))[:, :, 5:6]
    krec, mq, ms, ksym = kv.encode_keys(k, t)
    trec, tmq, tms, tsym = kv.encode_keys_tokenwise(k, t)
    assert np.array_equal(trec, krec[:, 0]) and np.array_equal(tsym, ksym[:, 0])
    assert np.array_equal(tmq, mq) and np.array_equal(tms.view(np.uint16), ms.view(np.uint16))
    vrec, vsym = kv.encode_values(v, t)
    tvrec, tvsym = kv.encode_values_tokenwise(v, t)
    assert np.array_equal(tvrec, vrec[:, 0]) and np.array_equal(tvsym, vsym[:, 0])


def test_token_streams_reconstruct_every_head():
    wl, tk, tv = _tabs()
    B, T, H, d = 1, 128, 8, 128
    k = wlmod.bf16_bits(wlmod.make_k(wl, 4, batch=B, context=T))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 4, batch=B, context=T))
    krec, mq, ms, ksym = kv.encode_keys_tokenwise(k, tk)
    vrec, vsym = kv.encode_values_tokenwise(v, tv)
    assert krec.shape == (B, T, 335) and vrec.shape == (B, T, 235) and mq.shape == (B, H, 1, d)
    for rec, sym, tab in ((krec, ksym, tk), (vrec, vsym, tv)):
        dsym, s16, o16, ok = kv.decode_records(rec, tab, H * d)
        assert ok.all() and np.array_equal(dsym, sym)
        assert np.all(tab.cost[sym].sum(axis=-1) <= tab.budget_q16)
    _, ks, ko, _ = kv.decode_records(krec, tk, H * d)
    _, vs, vo, _ = kv.decode_records(vrec, tv, H * d)
    sym_h, s_h, o_h = kv.tokenwise_as_heads(ksym, ks, ko, H)
    khat = attention.dequantize(sym_h, s_h, o_h, kmean.dequantize_mean(mq, ms))
    vsym_h, vs_h, vo_h = kv.tokenwise_as_heads(vsym, vs, vo, H)
    vhat = attention.dequantize(vsym_h, vs_h, vo_h)
    y_k = kv.rotate(k).transpose(0, 2, 1, 3)
    y_v = kv.rotate(v).transpose(0, 2, 1, 3)
    for y, yh, bound in ((y_k, khat, 0.15), (y_v, vhat, 0.25)):
        for h in range(H):
            e = ((y[:, h] - yh[:, h]) ** 2).sum() / ((y[:, h] - y[:, h].mean(axis=1, keepdims=True)) ** 2).sum()
            assert e < bound, (h, e)
        # a head shift (reading head h from the stream segment of h + 1) fails
        shifted = np.roll(yh, 1, axis=1)
        e = ((y - shifted) ** 2).sum() / ((y - y.mean(axis=2, keepdims=True)) ** 2).sum()
        assert e > 1.0


@pytest.mark.parametrize("p", [8, 12])
def test_default_operating_point_matches_table2(p):
    """N(0,1) tokens of 8 heads x 128 (rotation keeps them N(0,1)): key
    NMSE at M = 8 / 335 B and value NMSE at M = 6 / 235 B within 15 % of
    Tab. 2 (5.9 % and 14.1 %), with 8- and 12-bit tables."""
    tk = tables.build_tables(1024, 8, p, 1.4, 335)
    tv = tables.build_tables(1024, 6, p, 1.4, 235)
    rng = np.random.default_rng(7)
    x = rng.normal(size=(1, 96, 8, 128)).astype(np.float32)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)          # bf16 by truncation: still ~N(0, 1)
    y = kv.rotate(bits) / np.sqrt(128)                          # orthonormal rotation of N(0,1) is N(0,1)
    for tab, ref in ((tk, 5.9), (tv, 14.1)):
        xs = y.reshape(-1, 1024)
        _, sym, s16, o16, _ = kv.encode_streams(xs, tab)
        xh = s16.astype(np.float64)[:, None] * sym + o16.astype(np.float64)[:, None]
        nmse = 100 * ((xs - xh) ** 2).sum() / (xs ** 2).sum()
        assert abs(nmse / ref - 1) < 0.15, (tab.M, nmse)


def test_folded_attention_over_token_streams():
    wl, tk, tv = _tabs()
    B, T, H, G, d = 2, 128, 8, 4, 128
    k = wlmod.bf16_bits(wlmod.make_k(wl, 5, batch=B, context=T))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 5, batch=B, context=T))
    q = kv.bf16_to_f64(wlmod.bf16_bits(wlmod.make_q(wl, 5, batch=B)))
    krec, mq, ms, ksym = kv.encode_keys_tokenwise(k, tk)
    vrec, vsym = kv.encode_values_tokenwise(v, tv)
    _, ks, ko, _ = kv.decode_records(krec, tk, H * d)
    _, vs, vo, _ = kv.decode_records(vrec, tv, H * d)
    kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
    vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
    mean_hat = kmean.dequantize_mean(mq, ms)
    lens = [T, 77]
    scale = 1 / np.sqrt(d)
    a = attention.attention_folded(q, kh, ksh, koh, mean_hat, vh, vsh, voh, lens, G, scale)
    b = attention.attention_direct(q, attention.dequantize(kh, ksh, koh, mean_hat),
                                   attention.dequantize(vh, vsh, voh), lens, G, scale)
    assert np.max(np.abs(a - b)) < 1e-10 * np.max(np.abs(b))


def test_token_tables_need_h_times_d():
    wl, tk, _ = _tabs()
    k = wlmod.bf16_bits(wlmod.make_k(wl, 0, batch=1, context=128))[:, :, :4]
    with pytest.raises(ValueError):
        kv.encode_keys_tokenwise(k, tk)
