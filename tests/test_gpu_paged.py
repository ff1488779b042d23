"""Paged layout: records and key means in pool pages addressed through a block
table.  The paged calls must give exactly what the contiguous calls give
(bit-identical records, means and attention outputs: same arithmetic, only
the addresses differ), and the contiguous path is the one checked against
the oracle elsewhere; here it is re-checked against the oracle once more.
"""

import ctypes

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables

pytestmark = pytest.mark.gpu

DEV = "cuda"
TOL = 2e-3


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


def _setup(dq, page=256, max_pages=4, extra=5, seed=41):
    wl = wlmod.workload("b1_t4k")
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, G = 3, 2, 4
    t_cap = page * max_pages
    num_pages = B * max_pages + extra
    rng = np.random.default_rng(seed)
    bt = rng.permutation(num_pages)[: B * max_pages].reshape(B, max_pages).astype(np.int32)
    w2 = wlmod.Workload("paged", B, t_cap, Hkv * G, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, seed).to(DEV)
    v = wlmod.make_v(w2, seed).to(DEV)
    q = wlmod.make_q(w2, seed).to(DEV)
    return wl, gtk, gtv, B, Hkv, G, page, max_pages, t_cap, num_pages, bt, k, v, q


def _pools(num_pages, Hkv, page, wl):
    # one spare page past num_pages: every access through a valid entry stays
    # inside the first num_pages pages
    kp = torch.zeros((num_pages + 1, Hkv, page, wl.k.record_bytes), dtype=torch.uint8, device=DEV)
    vp = torch.zeros((num_pages + 1, Hkv, page, wl.v.record_bytes), dtype=torch.uint8, device=DEV)
    mq = torch.zeros((num_pages + 1, Hkv, page // 128, 128), dtype=torch.int8, device=DEV)
    ms = torch.zeros((num_pages + 1, Hkv, page // 128), dtype=torch.int16, device=DEV)
    return kp, vp, mq, ms


def test_paged_encode_and_attention_equal_contiguous(dq):
    wl, gtk, gtv, B, Hkv, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _setup(dq)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    # contiguous reference
    cache = dq.KVCache(B, Hkv, Hkv * G, t_cap, gtk, gtv, device=DEV)
    dq.dq_encode_kv(gtk, k[:, :512], 0, t_cap, cache.k_records, cache.k_mean_q, cache.k_mean_scale, status)
    dq.dq_encode_kv(gtk, k[:, 512:], 512, t_cap, cache.k_records, cache.k_mean_q, cache.k_mean_scale, status)
    dq.dq_encode_kv(gtv, v[:, :300], 0, t_cap, cache.v_records, None, None, status)
    dq.dq_encode_kv(gtv, v[:, 300:], 300, t_cap, cache.v_records, None, None, status)
    # paged, same appends (values start mid-tile and cross pages)
    kp, vp, mq, ms = _pools(num_pages, Hkv, page, wl)
    btd = torch.from_numpy(bt).to(DEV)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    dq.dq_encode_kv_paged(gtk, k[:, :512], 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_paged(gtk, k[:, 512:], 512, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_paged(gtv, v[:, :300], 0, btd, vpool, None, None, status)
    dq.dq_encode_kv_paged(gtv, v[:, 300:], 300, btd, vpool, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for b in range(B):
        for i in range(max_pages):
            p, sl = int(bt[b, i]), slice(i * page, (i + 1) * page)
            assert torch.equal(kpool[p], cache.k_records[b, :, sl])
            assert torch.equal(vpool[p], cache.v_records[b, :, sl])
            assert torch.equal(mqpool[p], cache.k_mean_q[b, :, i * page // 128:(i + 1) * page // 128])
            assert torch.equal(mspool[p], cache.k_mean_scale[b, :, i * page // 128:(i + 1) * page // 128])
    assert int(kp[num_pages].abs().sum()) == 0       # the spare page is never touched
    # attention: identical outputs
    lens = torch.tensor([t_cap, 0, 700], dtype=torch.int32, device=DEV)
    out_c = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    out_p = torch.empty_like(out_c)
    dq.dq_decode_attention(gtk, gtv, q, cache.k_records, cache.k_mean_q, cache.k_mean_scale, cache.v_records,
                           lens, out_c, cache.workspace, status=status)
    ws = torch.empty_like(cache.workspace)
    dq.dq_decode_attention_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btd, lens, ws, status=status)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, lens, t_cap, ws, out_p)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(out_c, out_p)
    # and the oracle on the same tokens
    otk = tables.build_tables(128, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(128, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    kb, vb = wlmod.bf16_bits(k.cpu()), wlmod.bf16_bits(v.cpu())
    krec, m_q, m_s, ksym = kv.encode_keys(kb, otk)
    vrec, vsym = kv.encode_values(vb, otv)
    _, ks, ko, _ = kv.decode_records(krec, otk, 128)
    _, vs, vo, _ = kv.decode_records(vrec, otv, 128)
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q.cpu())), ksym, ks, ko,
                                     kmean.dequantize_mean(m_q, m_s), vsym, vs, vo, lens.tolist(), G,
                                     1 / np.sqrt(128))
    got = out_p.cpu().numpy().astype(np.float64)
    live = [0, 2]
    scale = np.max(np.abs(ref[live]), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got[live] - ref[live]) / scale)) < TOL
    assert np.all(got[1] == 0.0)


def test_paged_bad_block_table_entry_is_flagged(dq):
    wl, gtk, gtv, B, Hkv, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _setup(dq, seed=42)
    kp, vp, mq, ms = _pools(num_pages, Hkv, page, wl)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    bad = bt.copy()
    bad[1, 2] = num_pages          # one past the pool
    btd = torch.from_numpy(bad).to(DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_encode_kv_paged(gtk, k, 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_paged(gtv, v, 0, btd, vpool, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_PAGE
    assert int(kp[num_pages].abs().sum()) == 0 and int(mq[num_pages].abs().sum()) == 0
    status.zero_()
    lens = torch.tensor([t_cap, t_cap, t_cap], dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    dq.dq_decode_attention_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btd, lens, ws, status=status)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, lens, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_PAGE
    assert torch.isfinite(out).all()


# ---- per-token records (one stream per token over all KV heads) in pages

def _token_setup(dq, page=256, max_pages=4, extra=5, seed=43, H=2, G=4, Ck=88, Cv=62, p=8):
    B = 3
    gtk = dq.Tables(128 * H, 8, p, Ck, 1.4)
    gtv = dq.Tables(128 * H, 6, p, Cv, 1.4)
    t_cap = page * max_pages
    num_pages = B * max_pages + extra
    rng = np.random.default_rng(seed)
    bt = rng.permutation(num_pages)[: B * max_pages].reshape(B, max_pages).astype(np.int32)
    wl = wlmod.workload("b1_t4k_tok")
    w2 = wlmod.Workload("tok_paged", B, t_cap, H * G, H, 4, wl.k, wl.v, streams="token")
    k = wlmod.make_k(w2, seed).to(DEV)
    v = wlmod.make_v(w2, seed).to(DEV)
    q = wlmod.make_q(w2, seed).to(DEV)
    return gtk, gtv, B, H, G, page, max_pages, t_cap, num_pages, bt, k, v, q


def _token_pools(dq, gtk, gtv, num_pages, H, page):
    # one spare page past num_pages, as above
    kp = torch.zeros(dq.token_pool_shape(gtk, num_pages + 1, page), dtype=torch.uint8, device=DEV)
    vp = torch.zeros(dq.token_pool_shape(gtv, num_pages + 1, page), dtype=torch.uint8, device=DEV)
    mq = torch.zeros((num_pages + 1, H, page // 128, 128), dtype=torch.int8, device=DEV)
    ms = torch.zeros((num_pages + 1, H, page // 128), dtype=torch.int16, device=DEV)
    return kp, vp, mq, ms


# (KV heads, query heads per KV head, K / V record bytes, p, page tokens, pages per sequence):
# a small stream, the paper's operating point (8 heads, 331 + 4 / 231 + 4 bytes)
# and p = 12 with two query heads per KV head
TOKEN_PAGED = [(2, 4, 88, 62, 8, 256, 4), (8, 4, 335, 235, 8, 128, 2), (4, 2, 170, 120, 12, 128, 4)]


@pytest.mark.parametrize("H,G,Ck,Cv,p,page,max_pages", TOKEN_PAGED)
def test_token_paged_encode_and_attention_equal_contiguous(dq, H, G, Ck, Cv, p, page, max_pages):
    gtk, gtv, B, H, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _token_setup(
        dq, page=page, max_pages=max_pages, H=H, G=G, Ck=Ck, Cv=Cv, p=p)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    cache = dq.TokenKVCache(B, H, H * G, t_cap, gtk, gtv, device=DEV)
    kh, vs = t_cap // 2, 300 * t_cap // 1024      # keys in whole windows, values mid-tile
    dq.dq_encode_kv_token(gtk, k[:, :kh], 0, t_cap, cache.k_records, cache.k_mean_q, cache.k_mean_scale, status)
    dq.dq_encode_kv_token(gtk, k[:, kh:], kh, t_cap, cache.k_records, cache.k_mean_q, cache.k_mean_scale, status)
    dq.dq_encode_kv_token(gtv, v[:, :vs], 0, t_cap, cache.v_records, None, None, status)
    dq.dq_encode_kv_token(gtv, v[:, vs:], vs, t_cap, cache.v_records, None, None, status)
    kp, vp, mq, ms = _token_pools(dq, gtk, gtv, num_pages, H, page)
    btd = torch.from_numpy(bt).to(DEV)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    dq.dq_encode_kv_token_paged(gtk, k[:, :kh], 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_token_paged(gtk, k[:, kh:], kh, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_token_paged(gtv, v[:, :vs], 0, btd, vpool, None, None, status)
    dq.dq_encode_kv_token_paged(gtv, v[:, vs:], vs, btd, vpool, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    tiles = page // 64
    for b in range(B):
        for i in range(max_pages):
            pp = int(bt[b, i])
            assert torch.equal(kpool[pp], cache.k_records[b, i * tiles:(i + 1) * tiles])
            assert torch.equal(vpool[pp], cache.v_records[b, i * tiles:(i + 1) * tiles])
            assert torch.equal(mqpool[pp], cache.k_mean_q[b, :, i * page // 128:(i + 1) * page // 128])
            assert torch.equal(mspool[pp], cache.k_mean_scale[b, :, i * page // 128:(i + 1) * page // 128])
    assert int(kp[num_pages].abs().sum()) == 0 and int(vp[num_pages].abs().sum()) == 0
    lens = torch.tensor([t_cap, 0, 700 * t_cap // 1024], dtype=torch.int32, device=DEV)
    out_c = cache.attend(q, lens)
    ws = torch.empty_like(cache.workspace)
    out_p = torch.empty_like(out_c)
    dq.dq_decode_attention_token_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btd, lens, ws,
                                               status=status)
    dq.dq_decode_attention_merge(B, H * G, H, lens, t_cap, ws, out_p)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(out_c, out_p)
    # and the oracle on the same tokens
    otk = tables.build_tables(128 * H, 8, p, 1.4, Ck)
    otv = tables.build_tables(128 * H, 6, p, 1.4, Cv)
    kb, vb = wlmod.bf16_bits(k.cpu()), wlmod.bf16_bits(v.cpu())
    krec, m_q, m_s, _ = kv.encode_keys_tokenwise(kb, otk)
    vrec, _ = kv.encode_values_tokenwise(vb, otv)
    ksym, ks, ko, _ = kv.decode_records(krec, otk, 128 * H)
    vsym, vs, vo, _ = kv.decode_records(vrec, otv, 128 * H)
    kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
    vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q.cpu())), kh, ksh, koh,
                                     kmean.dequantize_mean(m_q, m_s), vh, vsh, voh, lens.tolist(), G,
                                     1 / np.sqrt(128))
    got = out_p.cpu().numpy().astype(np.float64)
    live = [0, 2]
    scale = np.max(np.abs(ref[live]), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got[live] - ref[live]) / scale)) < TOL
    assert np.all(got[1] == 0.0)


def test_token_paged_bad_block_table_entry_is_flagged(dq):
    gtk, gtv, B, H, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _token_setup(dq, seed=44)
    kp, vp, mq, ms = _token_pools(dq, gtk, gtv, num_pages, H, page)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    bad = bt.copy()
    bad[1, 2] = num_pages          # one past the pool
    btd = torch.from_numpy(bad).to(DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_encode_kv_token_paged(gtk, k, 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_token_paged(gtv, v, 0, btd, vpool, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_PAGE
    assert int(kp[num_pages].abs().sum()) == 0 and int(mq[num_pages].abs().sum()) == 0
    status.zero_()
    lens = torch.tensor([t_cap, t_cap, t_cap], dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    dq.dq_decode_attention_token_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btd, lens, ws,
                                               status=status)
    dq.dq_decode_attention_merge(B, H * G, H, lens, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_PAGE
    assert torch.isfinite(out).all()


def test_token_paged_arguments_rejected(dq):
    gtk, gtv, B, H, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _token_setup(dq, seed=45)
    lib = dq._lib._lib
    kp, vp, mq, ms = _token_pools(dq, gtk, gtv, num_pages, H, page)
    btd = torch.from_numpy(bt).to(DEV)
    p = kp.data_ptr()

    def enc(page_tokens=page, num=num_pages, maxp=max_pages, tab=gtk, n_new=128):
        return lib.dq_encode_kv_token_paged(tab.handle, k.data_ptr(), k.stride(0), k.stride(1), k.stride(2), B, H,
                                            0, n_new, btd.data_ptr(), maxp, page_tokens, num, p, None, None, None,
                                            None)
    assert enc() == dq.DQ_OK
    assert enc(page_tokens=192) == dq.DQ_ERR_INVALID_ARG      # not a power of two
    assert enc(page_tokens=64) == dq.DQ_ERR_INVALID_ARG       # below a mean window
    assert enc(num=0) == dq.DQ_ERR_INVALID_ARG
    assert enc(maxp=0) == dq.DQ_ERR_INVALID_ARG
    assert enc(n_new=t_cap + 128) == dq.DQ_ERR_INVALID_ARG   # past the logical capacity
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, t_cap), dtype=torch.uint8, device=DEV)
    lens = torch.tensor([t_cap] * B, dtype=torch.int32, device=DEV)

    def attn(Hq=H * G, ws_bytes=ws.numel(), page_tokens=page):
        return lib.dq_decode_attention_token_paged_partial(gtk.handle, gtv.handle, q.data_ptr(), B, Hq, H, p,
                                                           mq.data_ptr(), ms.data_ptr(), vp.data_ptr(),
                                                           btd.data_ptr(), max_pages, page_tokens, num_pages,
                                                           lens.data_ptr(), ctypes.c_float(1 / 128 ** 0.5),
                                                           ws.data_ptr(), ws_bytes, None, None)
    assert attn(Hq=H * 16) == dq.DQ_ERR_INVALID_ARG          # at most 8 query heads per KV head
    assert attn(ws_bytes=64) == dq.DQ_ERR_WORKSPACE
    assert attn(page_tokens=100) == dq.DQ_ERR_INVALID_ARG
    torch.cuda.synchronize()


# ---- block tables whose entries past a sequence's length are unmapped (-1),
#      as serving engines leave them: a valid call, no status bit

def _unmap_past_length(bt, lens, page):
    out = bt.copy()
    for b, n in enumerate(lens):
        out[b, (n + page - 1) // page:] = -1
    return out


@pytest.mark.parametrize("lens_frac", [(1.0, 0.0, 0.68), (0.3, 0.55, 0.126)])
def test_paged_unmapped_tail_entries_are_not_read(dq, lens_frac):
    wl, gtk, gtv, B, Hkv, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _setup(dq, seed=46)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    cache = dq.KVCache(B, Hkv, Hkv * G, t_cap, gtk, gtv, device=DEV)
    cache.append(k, v, 0)
    kp, vp, mq, ms = _pools(num_pages, Hkv, page, wl)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    btd = torch.from_numpy(bt).to(DEV)
    dq.dq_encode_kv_paged(gtk, k, 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_paged(gtv, v, 0, btd, vpool, None, None, status)
    lens = [int(f * t_cap) for f in lens_frac]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out_c = cache.attend(q, seq)
    btu = torch.from_numpy(_unmap_past_length(bt, lens, page)).to(DEV)
    ws = torch.empty_like(cache.workspace)
    out_p = torch.empty_like(out_c)
    dq.dq_decode_attention_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btu, seq, ws, status=status)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out_p)
    torch.cuda.synchronize()
    assert int(status.item()) == 0 and int(cache.status.item()) == 0
    assert torch.equal(out_c, out_p)


@pytest.mark.parametrize("lens_frac", [(1.0, 0.0, 0.68), (0.3, 0.55, 0.126)])
def test_token_paged_unmapped_tail_entries_are_not_read(dq, lens_frac):
    gtk, gtv, B, H, G, page, max_pages, t_cap, num_pages, bt, k, v, q = _token_setup(dq, seed=47)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    cache = dq.TokenKVCache(B, H, H * G, t_cap, gtk, gtv, device=DEV)
    dq.dq_encode_kv_token(gtk, k, 0, t_cap, cache.k_records, cache.k_mean_q, cache.k_mean_scale, status)
    dq.dq_encode_kv_token(gtv, v, 0, t_cap, cache.v_records, None, None, status)
    kp, vp, mq, ms = _token_pools(dq, gtk, gtv, num_pages, H, page)
    kpool, vpool, mqpool, mspool = kp[:num_pages], vp[:num_pages], mq[:num_pages], ms[:num_pages]
    btd = torch.from_numpy(bt).to(DEV)
    dq.dq_encode_kv_token_paged(gtk, k, 0, btd, kpool, mqpool, mspool, status)
    dq.dq_encode_kv_token_paged(gtv, v, 0, btd, vpool, None, None, status)
    lens = [int(f * t_cap) for f in lens_frac]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out_c = cache.attend(q, seq)
    btu = torch.from_numpy(_unmap_past_length(bt, lens, page)).to(DEV)
    ws = torch.empty_like(cache.workspace)
    out_p = torch.empty_like(out_c)
    dq.dq_decode_attention_token_paged_partial(gtk, gtv, q, kpool, mqpool, mspool, vpool, btu, seq, ws,
                                               status=status)
    dq.dq_decode_attention_merge(B, H * G, H, seq, t_cap, ws, out_p)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(out_c, out_p)
