"""Prerotated tensors on the GPU (Sec. 4.2: values whose rotation is folded
into the projection weights; dq_config.prerotated), against the oracle's
readings V0 / A4, through the C ABI.

* Records and key means bit-exact with the oracle coding the tensor as it
  is (Gaussian inputs, values and keys, per (token, KV head) and per token).
* Ternary inputs, whose rotation is exact in bf16: the prerotated path on
  H x gives the online path's records on x bit for bit, and attention with
  the query given as H q / d and values as H v returns H times the online
  output (keys) / the online output (keys only prerotated).
* Attention within 2e-3 of the oracle, with a residual window whose raw
  tokens are in the same bases.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, hadamard, kmean, kv, tables
from tokrec import to_tiles

pytestmark = pytest.mark.gpu

DEV = "cuda"
TOL = 2e-3
D = 128


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


def _rel_err(got, ref):
    scale = np.maximum(np.max(np.abs(ref), axis=-1, keepdims=True), 1e-30)
    return float(np.max(np.abs(got - ref) / scale))


def _rotated_bf16(x_bf16):
    """H x of a bf16 tensor whose rotation is exact in bf16 (ternary input)."""
    h = hadamard.fwht(kv.bf16_to_f64(wlmod.bf16_bits(x_bf16)))
    t = torch.from_numpy(h.astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(t.float().numpy().astype(np.float64), h)
    return t


def _wl(B, T, H, G):
    base = wlmod.workload("b1_t4k")
    return wlmod.Workload("prerot", B, T, H * G, H, 4, base.k, base.v)


@pytest.mark.parametrize("pre_k,pre_v", [(False, True), (True, True), (True, False)])
def test_prerotated_gaussian_records_and_attention(dq, pre_k, pre_v):
    B, T, H, G = 3, 512, 2, 4
    wl = _wl(B, T, H, G)
    gtk = dq.Tables(D, 6, 12, 36, 1.4, prerotated=pre_k)
    gtv = dq.Tables(D, 6, 12, 36, 1.4, prerotated=pre_v)
    ot = tables.build_tables(D, 6, 12, 1.4, 36)
    k, v, q = wlmod.make_k(wl, 81), wlmod.make_v(wl, 81), wlmod.make_q(wl, 81)
    cache = dq.KVCache(B, H, H * G, T, gtk, gtv, device=DEV)
    cache.append(k.to(DEV), v.to(DEV), 0)
    lens = [T, 300, 0]
    out = cache.attend(q.to(DEV), torch.tensor(lens, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert int(cache.status.item()) == 0
    krec, mq, ms, ksym = kv.encode_keys(wlmod.bf16_bits(k), ot, rotate_on=not pre_k)
    vrec, vsym = kv.encode_values(wlmod.bf16_bits(v), ot, rotate_on=not pre_v)
    assert np.array_equal(cache.k_records.cpu().numpy(), krec)
    assert np.array_equal(cache.k_mean_q.cpu().numpy(), mq)
    assert np.array_equal(cache.k_mean_scale.cpu().numpy().view(np.uint16), ms.view(np.uint16))
    assert np.array_equal(cache.v_records.cpu().numpy(), vrec)
    _, ks, ko, _ = kv.decode_records(krec, ot, D)
    _, vs, vo, _ = kv.decode_records(vrec, ot, D)
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q)), ksym, ks, ko,
                                     kmean.dequantize_mean(mq, ms), vsym, vs, vo, lens, G, 1 / np.sqrt(D),
                                     rotate_k=not pre_k, rotate_v=not pre_v)
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(got[2] == 0)
    assert _rel_err(got[:2], ref[:2]) < TOL


def test_prerotated_ternary_equals_online_path(dq):
    B, T, H, G = 2, 384, 2, 4
    gtk, gtv = dq.Tables(D, 6, 12, 36, 1.4), dq.Tables(D, 6, 12, 36, 1.4)
    ptk = dq.Tables(D, 6, 12, 36, 1.4, prerotated=True)
    ptv = dq.Tables(D, 6, 12, 36, 1.4, prerotated=True)
    k = wlmod.make_ternary(91, B, T, H)
    v = wlmod.make_ternary(92, B, T, H)
    q = wlmod.make_ternary(93, B, H * G, 1)[:, :, 0].contiguous()
    hq = torch.from_numpy((hadamard.fwht(kv.bf16_to_f64(wlmod.bf16_bits(q))) / D).astype(np.float32))
    hq = hq.to(torch.bfloat16)                      # multiples of 1/128 below 1: exact
    on = dq.KVCache(B, H, H * G, T, gtk, gtv, device=DEV)
    on.append(k.to(DEV), v.to(DEV), 0)
    pre = dq.KVCache(B, H, H * G, T, ptk, ptv, device=DEV)
    pre.append(_rotated_bf16(k).to(DEV), _rotated_bf16(v).to(DEV), 0)
    mix = dq.KVCache(B, H, H * G, T, ptk, gtv, device=DEV)
    mix.append(_rotated_bf16(k).to(DEV), v.to(DEV), 0)
    lens = torch.tensor([T, 129], dtype=torch.int32, device=DEV)
    out_on = on.attend(q.to(DEV), lens)
    out_pre = pre.attend(hq.to(DEV), lens)
    out_mix = mix.attend(hq.to(DEV), lens)
    torch.cuda.synchronize()
    assert int(on.status.item()) == 0 and int(pre.status.item()) == 0 and int(mix.status.item()) == 0
    for name in ("k_records", "k_mean_q", "k_mean_scale", "v_records"):
        assert torch.equal(getattr(on, name), getattr(pre, name)), name
    a = out_on.cpu().numpy().astype(np.float64)
    assert _rel_err(out_pre.cpu().numpy().astype(np.float64), hadamard.fwht(a)) < TOL
    assert _rel_err(out_mix.cpu().numpy().astype(np.float64), a) < TOL


def test_prerotated_values_with_residual_window(dq):
    B, T, H, G, R = 2, 256, 2, 4, 256
    wl = _wl(B, T, H, G)
    gtk = dq.Tables(D, 6, 12, 36, 1.4)
    gtv = dq.Tables(D, 6, 12, 36, 1.4, prerotated=True)
    ot = tables.build_tables(D, 6, 12, 1.4, 36)
    k, v, q = wlmod.make_k(wl, 95), wlmod.make_v(wl, 95), wlmod.make_q(wl, 95)
    cache = dq.KVCache(B, H, H * G, T, gtk, gtv, device=DEV)
    cache.append(k.to(DEV), v.to(DEV), 0)
    g = torch.Generator().manual_seed(96)
    rk = torch.randn((B, H, R, D), generator=g).to(torch.bfloat16)
    rv = torch.randn((B, H, R, D), generator=g).to(torch.bfloat16)
    seq_l, res_l = [T, 128], [70, 200]
    seq = torch.tensor(seq_l, dtype=torch.int32, device=DEV)
    res = torch.tensor(res_l, dtype=torch.int32, device=DEV)
    qd = q.to(DEV)
    out = torch.empty((B, H * G, D), dtype=torch.float32, device=DEV)
    cache.partial(qd, seq)
    dq.dq_decode_attention_residual(qd, rk.to(DEV), rv.to(DEV), seq, res, T, cache.workspace)
    cache.merge(seq, out)
    torch.cuda.synchronize()
    assert int(cache.status.item()) == 0
    krec, mq, ms, ksym = kv.encode_keys(wlmod.bf16_bits(k), ot)
    vrec, vsym = kv.encode_values(wlmod.bf16_bits(v), ot, rotate_on=False)
    _, ks, ko, _ = kv.decode_records(krec, ot, D)
    _, vs, vo, _ = kv.decode_records(vrec, ot, D)
    k_rot = attention.dequantize(ksym, ks, ko, kmean.dequantize_mean(mq, ms))
    v_rot = attention.dequantize(vsym, vs, vo)
    # ring slot of residual token i: (seq_len + i) mod R
    rk64, rv64 = kv.bf16_to_f64(wlmod.bf16_bits(rk)), kv.bf16_to_f64(wlmod.bf16_bits(rv))
    rk_o = np.stack([np.roll(rk64[b], -seq_l[b] % R, axis=1) for b in range(B)])
    rv_o = np.stack([np.roll(rv64[b], -seq_l[b] % R, axis=1) for b in range(B)])
    ref = attention.attention_with_residual(kv.bf16_to_f64(wlmod.bf16_bits(q)), k_rot, v_rot, seq_l, rk_o, rv_o,
                                            res_l, G, 1 / np.sqrt(D), rotate_v=False)
    assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL
    # the one-launch window + merge over the same chunk partials
    out1 = torch.empty_like(out)
    dq.dq_decode_attention_merge_residual(qd, rk.to(DEV), rv.to(DEV), seq, res, T, cache.workspace, out1)
    torch.cuda.synchronize()
    assert _rel_err(out1.cpu().numpy().astype(np.float64), ref) < TOL
    assert _rel_err(out1.cpu().numpy().astype(np.float64), out.cpu().numpy().astype(np.float64)) < 1e-5


def test_prerotated_per_token_streams(dq):
    B, T, H, G = 2, 256, 4, 2
    n = D * H
    gtk = dq.Tables(n, 8, 8, 170, 1.4)
    gtv = dq.Tables(n, 6, 8, 120, 1.4, prerotated=True)
    otk, otv = tables.build_tables(n, 8, 8, 1.4, 170), tables.build_tables(n, 6, 8, 1.4, 120)
    wl = wlmod.Workload("prerot_tok", B, T, H * G, H, 4, wlmod.workload("b1_t4k").k, wlmod.workload("b1_t4k").v,
                        streams="token")
    k, v, q = wlmod.make_k(wl, 97), wlmod.make_v(wl, 97), wlmod.make_q(wl, 97)
    cache = dq.TokenKVCache(B, H, H * G, T, gtk, gtv, device=DEV)
    cache.append(k.to(DEV), v.to(DEV), 0)
    lens = [T, 100]
    out = cache.attend(q.to(DEV), torch.tensor(lens, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert int(cache.status.item()) == 0
    krec, mq, ms, _ = kv.encode_keys_tokenwise(wlmod.bf16_bits(k), otk)
    vrec, _ = kv.encode_values_tokenwise(wlmod.bf16_bits(v), otv, rotate_on=False)
    Sv = dq.dq_token_record_stride(gtv)
    assert np.array_equal(cache.v_records.cpu().numpy(), to_tiles(vrec, Sv))
    ksym, ks, ko, _ = kv.decode_records(krec, otk, n)
    vsym, vs, vo, _ = kv.decode_records(vrec, otv, n)
    kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
    vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q)), kh, ksh, koh,
                                     kmean.dequantize_mean(mq, ms), vh, vsh, voh, lens, G, 1 / np.sqrt(D),
                                     rotate_v=False)
    assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL


def test_prerotated_flag_validated(dq):
    import ctypes
    lib = dq._lib
    cfg = lib._Config(D, 6, 12, 36, 1.4, 2)
    h = ctypes.c_void_p()
    info = lib._Info()
    assert lib._lib.dq_build_tables(ctypes.byref(cfg), ctypes.byref(h), ctypes.byref(info)) == dq.DQ_ERR_INVALID_ARG
