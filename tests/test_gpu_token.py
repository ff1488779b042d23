"""Per-token streams (one stream of 128 H values per token over all KV heads,
the paper's default grouping) on the GPU against the oracle, through the C ABI.

Bars as in test_gpu_parity.py: records (first C bytes, then zero padding to
the 16-byte slot; buffers in 64-token tiles with 8-byte chunks outermost) and
key means bit-exact with the oracle's
encode_*_tokenwise; attention within 2e-3 (row-normalized) of the oracle's
fp64 folded attention over the oracle's own records, which are uploaded for
the attention checks.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables
from tokrec import from_tiles, to_tiles

pytestmark = pytest.mark.gpu

TOL = 2e-3
DEV = "cuda"


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


def _tabs(dq, n, levels, C, p=12, alpha=1.4):
    return dq.Tables(n, levels, p, C, alpha), tables.build_tables(n, levels, p, alpha, C)


def _rel_err(got, ref):
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    return float(np.max(np.abs(got - ref) / np.maximum(scale, 1e-30)))


def _oracle_attention(q_bits, krec, mq, ms, vrec, otk, otv, lens, H, G):
    n = 128 * H
    ksym, ks, ko, okk = kv.decode_records(krec, otk, n)
    vsym, vs, vo, okv = kv.decode_records(vrec, otv, n)
    assert okk.all() and okv.all()
    kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
    vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
    return attention.attention_folded(kv.bf16_to_f64(q_bits), kh, ksh, koh, kmean.dequantize_mean(mq, ms),
                                      vh, vsh, voh, lens, G, 1 / np.sqrt(128))


def _inputs(H, G, B, T, seed):
    wl = wlmod.workload("b1_t4k_tok")
    w2 = wlmod.Workload("tok", B, T, H * G, H, 4, wl.k, wl.v, streams="token")
    return wlmod.make_k(w2, seed), wlmod.make_v(w2, seed), wlmod.make_q(w2, seed)


@pytest.mark.parametrize("p", [12, 8])
def test_token_encode_bit_exact(dq, p):
    H, B, T = 8, 2, 256
    gtk, otk = _tabs(dq, 1024, 8, 335, p)
    gtv, otv = _tabs(dq, 1024, 6, 235, p)
    k, v, _ = _inputs(H, 4, B, T, 31)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(wlmod.bf16_bits(k), otk)
    vrec, _ = kv.encode_values_tokenwise(wlmod.bf16_bits(v), otv)
    Sk, Sv = dq.dq_token_record_stride(gtk), dq.dq_token_record_stride(gtv)
    assert (Sk, Sv) == (336, 240)
    # pad bytes must be rewritten
    grk = torch.full(dq.token_records_shape(gtk, B, T), 0xAB, dtype=torch.uint8, device=DEV)
    grv = torch.full(dq.token_records_shape(gtv, B, T), 0xAB, dtype=torch.uint8, device=DEV)
    gmq = torch.zeros((B, H, T // 128, 128), dtype=torch.int8, device=DEV)
    gms = torch.zeros((B, H, T // 128), dtype=torch.int16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    # appends: keys in whole windows, values at a ragged offset
    dq.dq_encode_kv_token(gtk, kd[:, :128], 0, T, grk, gmq, gms, status)
    dq.dq_encode_kv_token(gtk, kd[:, 128:], 128, T, grk, gmq, gms, status)
    dq.dq_encode_kv_token(gtv, vd[:, :100], 0, T, grv, None, None, status)
    dq.dq_encode_kv_token(gtv, vd[:, 100:], 100, T, grv, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert np.array_equal(grk.cpu().numpy(), to_tiles(krec, Sk))
    assert np.array_equal(grv.cpu().numpy(), to_tiles(vrec, Sv))
    assert np.array_equal(gmq.cpu().numpy(), mq)
    assert np.array_equal(gms.cpu().numpy().view(np.uint16), ms.view(np.uint16))


def _pad_tok(grk, gmq, gms, grv, cap):
    """The same cache in buffers of capacity cap (zero tiles past the old
    one).  The chunk plan follows the capacity: small capacities give chunks
    of at most 4 tiles, whose keys and values separate wavefronts decode; a
    capacity of 64 x 1024 tokens per sequence gives larger chunks, decoded
    with both chains in one wavefront."""
    def pad(x, n):
        shape = list(x.shape)
        shape[1 if x.dim() == 5 else 2] = n
        y = torch.zeros(shape, dtype=x.dtype, device=x.device)
        if x.dim() == 5:
            y[:, :x.shape[1]] = x
        else:
            y[:, :, :x.shape[2]] = x
        return y
    return pad(grk, cap // 64), pad(gmq, cap // 128), pad(gms, cap // 128), pad(grv, cap // 64)


@pytest.mark.parametrize("p,cap", [(12, None), (8, None), (8, 65536)])
def test_token_attention_matches_oracle(dq, p, cap):
    H, G, B, T = 8, 4, 4, 384
    gtk, otk = _tabs(dq, 1024, 8, 335, p)
    gtv, otv = _tabs(dq, 1024, 6, 235, p)
    k, v, q = _inputs(H, G, B, T, 32)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(wlmod.bf16_bits(k), otk)
    vrec, _ = kv.encode_values_tokenwise(wlmod.bf16_bits(v), otv)
    Sk, Sv = dq.dq_token_record_stride(gtk), dq.dq_token_record_stride(gtv)
    lens = [T, 0, 65, 300]
    grk = torch.from_numpy(to_tiles(krec, Sk)).to(DEV)
    grv = torch.from_numpy(to_tiles(vrec, Sv)).to(DEV)
    gmq = torch.from_numpy(mq).to(DEV)
    gms = torch.from_numpy(ms.view(np.int16)).to(DEV)
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    if cap is not None:
        grk, gmq, gms, grv = _pad_tok(grk, gmq, gms, grv, cap)
    tc = cap or T
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, tc), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_token_partial(gtk, gtv, qd, grk, gmq, gms, grv, seq, ws, status=status)
    dq.dq_decode_attention_merge(B, H * G, H, seq, tc, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    ref = _oracle_attention(wlmod.bf16_bits(q), krec, mq, ms, vrec, otk, otv, lens, H, G)
    assert np.all(got[1] == 0.0)
    live = [0, 2, 3]
    assert _rel_err(got[live], ref[live]) < TOL


@pytest.mark.parametrize("H,G,Ck,Cv,cap", [(8, 1, 335, 235, None), (4, 2, 170, 120, None), (2, 4, 88, 62, None),
                                           (1, 4, 44, 32, None), (8, 8, 335, 235, None), (4, 6, 170, 120, None),
                                           (2, 8, 88, 62, None), (1, 5, 44, 32, None),
                                           (8, 1, 335, 235, 131072), (2, 4, 88, 62, 131072)])
def test_token_attention_heads_and_groups(dq, H, G, Ck, Cv, cap):
    """Streams of 128 H values for H = 8, 4, 2, 1 KV heads and 1 to 8 query
    heads per KV head (above 4: two groups of query-head slots per KV head);
    the GPU encoder fills the cache.  Up to 4 query heads, also in buffers of
    131072 tokens (chunks of more than 4 tiles: both chains in one
    wavefront)."""
    B, T = 2, 256
    n = 128 * H
    gtk, otk = _tabs(dq, n, 8, Ck)
    gtv, otv = _tabs(dq, n, 6, Cv)
    assert otk.feasible and otv.feasible
    k, v, q = _inputs(H, G, B, T, 33 + H)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(wlmod.bf16_bits(k), otk)
    vrec, _ = kv.encode_values_tokenwise(wlmod.bf16_bits(v), otv)
    Sk, Sv = dq.dq_token_record_stride(gtk), dq.dq_token_record_stride(gtv)
    grk = torch.empty(dq.token_records_shape(gtk, B, T), dtype=torch.uint8, device=DEV)
    grv = torch.empty(dq.token_records_shape(gtv, B, T), dtype=torch.uint8, device=DEV)
    gmq = torch.empty((B, H, T // 128, 128), dtype=torch.int8, device=DEV)
    gms = torch.empty((B, H, T // 128), dtype=torch.int16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_encode_kv_token(gtk, k.to(DEV), 0, T, grk, gmq, gms, status)
    dq.dq_encode_kv_token(gtv, v.to(DEV), 0, T, grv, None, None, status)
    lens = [T, 129]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    assert np.array_equal(grk.cpu().numpy(), to_tiles(krec, Sk))
    assert np.array_equal(grv.cpu().numpy(), to_tiles(vrec, Sv))
    if cap is not None:
        grk, gmq, gms, grv = _pad_tok(grk, gmq, gms, grv, cap)
    tc = cap or T
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, tc), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    dq.dq_decode_attention_token_partial(gtk, gtv, q.to(DEV), grk, gmq, gms, grv, seq, ws, status=status)
    dq.dq_decode_attention_merge(B, H * G, H, seq, tc, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ref = _oracle_attention(wlmod.bf16_bits(q), krec, mq, ms, vrec, otk, otv, lens, H, G)
    assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL


@pytest.mark.parametrize("cap", [None, 65536])
def test_token_attention_flags_corrupt_record_and_is_deterministic(dq, cap):
    H, G, B, T = 8, 4, 2, 256
    gtk, otk = _tabs(dq, 1024, 8, 335)
    gtv, otv = _tabs(dq, 1024, 6, 235)
    k, v, q = _inputs(H, G, B, T, 34)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(wlmod.bf16_bits(k), otk)
    vrec, _ = kv.encode_values_tokenwise(wlmod.bf16_bits(v), otv)
    Sk, Sv = dq.dq_token_record_stride(gtk), dq.dq_token_record_stride(gtv)
    grk = torch.from_numpy(to_tiles(krec, Sk)).to(DEV)
    grv = torch.from_numpy(to_tiles(vrec, Sv)).to(DEV)
    gmq = torch.from_numpy(mq).to(DEV)
    gms = torch.from_numpy(ms.view(np.int16)).to(DEV)
    if cap is not None:
        grk, gmq, gms, grv = _pad_tok(grk, gmq, gms, grv, cap)
    T = cap or T
    seq = torch.tensor([256, 200], dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, T), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
        status = torch.zeros(1, dtype=torch.int32, device=DEV)
        dq.dq_decode_attention_token_partial(gtk, gtv, q.to(DEV), grk, gmq, gms, grv, seq, ws, status=status)
        dq.dq_decode_attention_merge(B, H * G, H, seq, T, ws, out)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1])
    # a record past the length is never read as a token: still clean
    bad = grv.clone()
    bad[1, 230 // 64, 0, 230 % 64, 4:8] = 0          # the state word of token 230
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_decode_attention_token_partial(gtk, gtv, q.to(DEV), grk, gmq, gms, bad, seq, ws, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    # a stream state that is not a valid end state inside the length: flagged,
    # outputs still finite
    bad[0, 0, 0, 17, 4:8] = 0
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    dq.dq_decode_attention_token_partial(gtk, gtv, q.to(DEV), grk, gmq, gms, bad, seq, ws, status=status)
    dq.dq_decode_attention_merge(B, H * G, H, seq, T, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_CORRUPT
    assert torch.isfinite(out).all()


def test_token_entry_points_reject_bad_arguments(dq):
    H, G, B, T = 8, 4, 1, 256
    gtk, _ = _tabs(dq, 1024, 8, 335)
    gtv, _ = _tabs(dq, 1024, 6, 235)
    g128 = dq.Tables(128, 6, 12, 36, 1.4)
    lib = dq._lib._lib
    big = torch.zeros(1 << 22, dtype=torch.uint8, device=DEV)
    p = big.data_ptr()

    def attn(tk, tv, Hq=H * G, Hkv=H, t_cap=T, ws_bytes=1 << 22):
        return lib.dq_decode_attention_token_partial(tk.handle, tv.handle, p, B, Hq, Hkv, p, p, p, p, p, t_cap,
                                                     0.088, p, ws_bytes, p, None)

    assert attn(g128, gtv) == dq.DQ_ERR_INVALID_ARG             # n must be 128 H
    assert attn(gtk, gtv, Hq=128) == dq.DQ_ERR_INVALID_ARG      # at most 8 query heads per KV head
    assert attn(gtk, gtv, Hq=30) == dq.DQ_ERR_INVALID_ARG       # not a multiple of H
    assert attn(gtk, gtv, t_cap=200) == dq.DQ_ERR_INVALID_ARG
    assert attn(gtk, gtv, ws_bytes=16) == dq.DQ_ERR_WORKSPACE
    rc = lib.dq_encode_kv_token(gtk.handle, p, 0, 128 * H, 128, B, 4, 0, 128, T, p, p, p, p, None)
    assert rc == dq.DQ_ERR_INVALID_ARG                          # 4 heads do not make n = 1024
    assert lib.dq_token_record_stride(None) == 0


def test_token_streams_with_residual_window(dq):
    """The paper's serving configuration (Sec. 5.1): per-token streams for the
    compressed tokens plus the newest tokens raw in BF16.  Per-token partial +
    residual partial + merge against the oracle's attention over the token-wise
    reconstructions and the raw tokens (reading A3)."""
    H, G, B, t_cap, r_cap = 8, 4, 3, 384, 256
    gtk, otk = _tabs(dq, 1024, 8, 335, 8)
    gtv, otv = _tabs(dq, 1024, 6, 235, 8)
    comp = [256, 0, 128]                      # compressed tokens (whole windows)
    res = [128, 40, 0]                        # raw tokens after them
    T = max(c + r for c, r in zip(comp, res))
    k, v, q = _inputs(H, G, B, T, 36)
    kb, vb = wlmod.bf16_bits(k), wlmod.bf16_bits(v)
    grk = torch.zeros(dq.token_records_shape(gtk, B, t_cap), dtype=torch.uint8, device=DEV)
    grv = torch.zeros(dq.token_records_shape(gtv, B, t_cap), dtype=torch.uint8, device=DEV)
    gmq = torch.zeros((B, H, t_cap // 128, 128), dtype=torch.int8, device=DEV)
    gms = torch.zeros((B, H, t_cap // 128), dtype=torch.int16, device=DEV)
    rk = torch.zeros((B, H, r_cap, 128), dtype=torch.bfloat16, device=DEV)
    rv = torch.zeros_like(rk)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    for b in range(B):
        n = comp[b]
        if n:
            dq.dq_encode_kv_token(gtk, kd[b:b + 1, :n], 0, t_cap, grk[b:b + 1], gmq[b:b + 1], gms[b:b + 1], status)
            dq.dq_encode_kv_token(gtv, vd[b:b + 1, :n], 0, t_cap, grv[b:b + 1], None, None, status)
        for i in range(res[b]):
            rk[b, :, (n + i) % r_cap] = kd[b, n + i]
            rv[b, :, (n + i) % r_cap] = vd[b, n + i]
    seq = torch.tensor(comp, dtype=torch.int32, device=DEV)
    rl = torch.tensor(res, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_token_partial(gtk, gtv, qd, grk, gmq, gms, grv, seq, ws, status=status)
    dq.dq_decode_attention_residual(qd, rk, rv, seq, rl, t_cap, ws)
    dq.dq_decode_attention_merge(B, H * G, H, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    # oracle: token-wise reconstruction of the compressed tokens, raw residual tokens
    Tc = max(comp)
    k_rot = np.zeros((B, H, Tc, 128))
    v_rot = np.zeros((B, H, Tc, 128))
    res_k = np.zeros((B, H, max(res), 128))
    res_v = np.zeros((B, H, max(res), 128))
    for b in range(B):
        n = comp[b]
        if n:
            krec, mq, ms, ksym = kv.encode_keys_tokenwise(kb[b:b + 1, :n], otk)
            vrec, vsym = kv.encode_values_tokenwise(vb[b:b + 1, :n], otv)
            _, ks, ko, _ = kv.decode_records(krec, otk, 1024)
            _, vs, vo, _ = kv.decode_records(vrec, otv, 1024)
            kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
            vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
            k_rot[b, :, :n] = attention.dequantize(kh, ksh, koh, kmean.dequantize_mean(mq, ms))[0]
            v_rot[b, :, :n] = attention.dequantize(vh, vsh, voh)[0]
        r = res[b]
        res_k[b, :, :r] = np.moveaxis(kv.bf16_to_f64(kb[b, n:n + r]), 0, 1)
        res_v[b, :, :r] = np.moveaxis(kv.bf16_to_f64(vb[b, n:n + r]), 0, 1)
    ref = attention.attention_with_residual(kv.bf16_to_f64(wlmod.bf16_bits(q)), k_rot, v_rot, comp, res_k, res_v,
                                            res, G, 1 / np.sqrt(128))
    assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL
    # the one-launch window + merge over the same chunk partials
    out1 = torch.empty_like(out)
    dq.dq_decode_attention_merge_residual(qd, rk, rv, seq, rl, t_cap, ws, out1)
    torch.cuda.synchronize()
    assert _rel_err(out1.cpu().numpy().astype(np.float64), ref) < TOL


def _oracle_stream(q_bits, kb, vb, comp, res, otk, otv, H, G):
    """Oracle attention over `comp` encoded tokens (token-wise streams, as the
    cache flushes them) followed by `res` raw tokens, the same for every
    sequence."""
    B = kb.shape[0]
    k_rot = np.zeros((B, H, max(comp, 1), 128))
    v_rot = np.zeros((B, H, max(comp, 1), 128))
    if comp:
        krec, mq, ms, ksym = kv.encode_keys_tokenwise(kb[:, :comp], otk)
        vrec, vsym = kv.encode_values_tokenwise(vb[:, :comp], otv)
        _, ks, ko, _ = kv.decode_records(krec, otk, 128 * H)
        _, vs, vo, _ = kv.decode_records(vrec, otv, 128 * H)
        kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
        vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
        k_rot[:, :, :comp] = attention.dequantize(kh, ksh, koh, kmean.dequantize_mean(mq, ms))
        v_rot[:, :, :comp] = attention.dequantize(vh, vsh, voh)
    res_k = np.moveaxis(kv.bf16_to_f64(kb[:, comp:comp + res]), 1, 2)
    res_v = np.moveaxis(kv.bf16_to_f64(vb[:, comp:comp + res]), 1, 2)
    return attention.attention_with_residual(kv.bf16_to_f64(q_bits), k_rot, v_rot, [comp] * B, res_k, res_v,
                                             [res] * B, G, 1 / np.sqrt(128))


def test_streaming_cache_over_token_streams(dq):
    """Serving semantics (Sec. 5.1) with the paper's per-token streams: a
    prefill, then one decode token at a time through the BF16 ring, each full
    window flushed into per-token records.  At several lengths the step
    (per-token partial + residual partial + merge) matches the oracle's
    attention over the token-wise reconstructions of the flushed tokens and
    the raw ring tokens; at the end the records and key means are the
    oracle's, bit for bit."""
    H, G, B, t_cap = 2, 4, 2, 1024
    gtk, otk = _tabs(dq, 128 * H, 8, 88, 8)
    gtv, otv = _tabs(dq, 128 * H, 6, 62, 8)
    prefill, steps = 300, 300
    T = prefill + steps
    k, v, _ = _inputs(H, G, B, T, 41)
    kb, vb = wlmod.bf16_bits(k), wlmod.bf16_bits(v)
    kd, vd = k.to(DEV), v.to(DEV)
    cache = dq.StreamingKVCache(B, H, H * G, t_cap, gtk, gtv, streams="token")
    cache.prefill(kd[:, :prefill], vd[:, :prefill])
    checks = {prefill, prefill + 84, prefill + 85, T}
    for t in range(prefill, T + 1):
        if t in checks:
            q = _inputs(H, G, B, 128, 1000 + t)[2]
            out = cache.attend(q.to(DEV))
            torch.cuda.synchronize()
            assert int(cache.status.item()) == 0
            comp, res = cache.n_comp, cache.n_res
            assert comp + res == t and comp % 128 == 0 and res >= min(t, 128)
            assert cache.seq_lens.tolist() == [comp] * B and cache.res_lens.tolist() == [res] * B
            ref = _oracle_stream(wlmod.bf16_bits(q), kb, vb, comp, res, otk, otv, H, G)
            assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL, t
        if t < T:
            cache.append(kd[:, t].contiguous(), vd[:, t].contiguous())
    n = cache.n_comp
    krec, mq, ms, _ = kv.encode_keys_tokenwise(kb[:, :n], otk)
    vrec, _ = kv.encode_values_tokenwise(vb[:, :n], otv)
    gk = from_tiles(cache.cache.k_records.cpu().numpy())
    gv = from_tiles(cache.cache.v_records.cpu().numpy())
    assert np.array_equal(gk[:, :n, :krec.shape[2]], krec) and not gk[:, :n, krec.shape[2]:].any()
    assert np.array_equal(gv[:, :n, :vrec.shape[2]], vrec) and not gv[:, :n, vrec.shape[2]:].any()
    assert np.array_equal(cache.cache.k_mean_q[:, :, :n // 128].cpu().numpy(), mq)
    assert np.array_equal(cache.cache.k_mean_scale[:, :, :n // 128].cpu().numpy().view(np.uint16),
                          ms.view(np.uint16))
