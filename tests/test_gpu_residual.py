"""Residual BF16 window (Sec. 5.1: the most recent tokens stay in BF16) on the
GPU against the oracle's attention over compressed + raw tokens.

Bars as in test_gpu_parity.py: records and key means bit-exact with the
oracle's own encoding of the same raw windows; attention within 2e-3
(row-normalized) of the oracle's fp64 attention over the oracle's
reconstructions plus the raw residual tokens.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables

pytestmark = pytest.mark.gpu

TOL = 2e-3
DEV = "cuda"


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


def _rel_err(got, ref):
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    return float(np.max(np.abs(got - ref) / np.maximum(scale, 1e-30)))


def _fused(dq, qd, res_k, res_v, seq, rl, t_cap, ws, two_call):
    """The one-launch window + merge over the chunk partials already in ws:
    returns its output; it must equal the two-call form up to fp32 rounding
    order (the window's sum skips the H, H / d round trip)."""
    out = torch.full(tuple(two_call.shape), float("nan"), dtype=torch.float32, device=DEV)
    dq.dq_decode_attention_merge_residual(qd, res_k, res_v, seq, rl, t_cap, ws, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    assert _rel_err(got, two_call) < 1e-5
    return got


def _oracle(q_bits, k_bits, v_bits, comp_lens, res_lens, otk, otv, G):
    """Oracle attention for sequences whose first comp_lens[b] tokens are
    encoded (window by window, as the cache does) and whose next res_lens[b]
    tokens are raw."""
    B, T, H, d = k_bits.shape
    Tc = max(comp_lens) if max(comp_lens) > 0 else 0
    Tc = -(-Tc // 128) * 128
    R = max(res_lens) if max(res_lens) > 0 else 1
    k_rot = np.zeros((B, H, max(Tc, 1), d))
    v_rot = np.zeros((B, H, max(Tc, 1), d))
    res_k = np.zeros((B, H, R, d))
    res_v = np.zeros((B, H, R, d))
    for b in range(B):
        n = comp_lens[b]
        if n:
            krec, mq, ms, _ = kv.encode_keys(k_bits[b:b + 1, :n], otk)
            vrec, _ = kv.encode_values(v_bits[b:b + 1, :n], otv)
            ks, kss, kso, _ = kv.decode_records(krec, otk, d)
            vs, vss, vso, _ = kv.decode_records(vrec, otv, d)
            k_rot[b, :, :n] = attention.dequantize(ks, kss, kso, kmean.dequantize_mean(mq, ms))[0]
            v_rot[b, :, :n] = attention.dequantize(vs, vss, vso)[0]
        r = res_lens[b]
        res_k[b, :, :r] = np.moveaxis(kv.bf16_to_f64(k_bits[b, n:n + r]), 0, 1)
        res_v[b, :, :r] = np.moveaxis(kv.bf16_to_f64(v_bits[b, n:n + r]), 0, 1)
    return attention.attention_with_residual(kv.bf16_to_f64(q_bits), k_rot, v_rot, comp_lens, res_k, res_v,
                                             res_lens, G, 1 / np.sqrt(d))


def test_attention_over_ring_and_compressed_tokens(dq):
    wl = wlmod.workload("b1_t4k")
    otk = tables.build_tables(128, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(128, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, G, t_cap, r_cap = 5, 2, 4, 512, 256
    comp = [384, 0, 256, 0, 128]          # compressed tokens (whole windows, as flushed)
    res = [200, 77, 0, 0, 256]            # ring wraps for sequences 0 and 4
    T = max(c + r for c, r in zip(comp, res))
    w2 = wlmod.Workload("ring", B, T, Hkv * G, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, 21)
    v = wlmod.make_v(w2, 21)
    q = wlmod.make_q(w2, 21)
    kb, vb, qb = wlmod.bf16_bits(k), wlmod.bf16_bits(v), wlmod.bf16_bits(q)

    records_k = torch.zeros((B, Hkv, t_cap, wl.k.record_bytes), dtype=torch.uint8, device=DEV)
    records_v = torch.zeros((B, Hkv, t_cap, wl.v.record_bytes), dtype=torch.uint8, device=DEV)
    mean_q = torch.zeros((B, Hkv, t_cap // 128, 128), dtype=torch.int8, device=DEV)
    mean_s = torch.zeros((B, Hkv, t_cap // 128), dtype=torch.int16, device=DEV)
    res_k = torch.zeros((B, Hkv, r_cap, 128), dtype=torch.bfloat16, device=DEV)
    res_v = torch.zeros_like(res_k)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    for b in range(B):
        n = comp[b]
        if n:
            dq.dq_encode_kv(gtk, kd[b:b + 1, :n], 0, t_cap, records_k[b:b + 1], mean_q[b:b + 1], mean_s[b:b + 1],
                            status)
            dq.dq_encode_kv(gtv, vd[b:b + 1, :n], 0, t_cap, records_v[b:b + 1], None, None, status)
        for i in range(res[b]):
            slot = (n + i) % r_cap
            res_k[b, :, slot] = kd[b, n + i]
            res_v[b, :, slot] = vd[b, n + i]
    seq = torch.tensor(comp, dtype=torch.int32, device=DEV)
    rl = torch.tensor(res, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_partial(gtk, gtv, qd, records_k, mean_q, mean_s, records_v, seq, ws, status=status)
    dq.dq_decode_attention_residual(qd, res_k, res_v, seq, rl, t_cap, ws)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    ref = _oracle(qb, kb, vb, comp, res, otk, otv, G)
    assert np.all(got[3] == 0.0)          # neither compressed nor residual tokens
    live = [0, 1, 2, 4]
    assert _rel_err(got[live], ref[live]) < TOL
    fused = _fused(dq, qd, res_k, res_v, seq, rl, t_cap, ws, got)
    assert np.all(fused[3] == 0.0)
    assert _rel_err(fused[live], ref[live]) < TOL

    # without the residual call the same workspace attends over the compressed tokens only
    dq.dq_decode_attention_partial(gtk, gtv, qd, records_k, mean_q, mean_s, records_v, seq, ws, status=status)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref0 = _oracle(qb, kb, vb, comp, [0] * B, otk, otv, G)
    assert np.all(got[[1, 3]] == 0.0)
    assert _rel_err(got[[0, 2, 4]], ref0[[0, 2, 4]]) < TOL


@pytest.mark.parametrize("G", [1, 2, 8])
def test_residual_query_groups(dq, G):
    """1, 2 and 8 query heads per KV head; residual lengths that give every
    part an odd count, one token, or halves of 1..32 tokens per wavefront."""
    wl = wlmod.workload("b1_t4k")
    otk = tables.build_tables(128, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(128, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, t_cap, r_cap = 6, 2, 256, 256
    comp = [128, 0, 256, 128, 0, 256]
    res = [255, 1, 5, 64, 129, 0]
    T = max(c + r for c, r in zip(comp, res))
    w2 = wlmod.Workload("ring_g", B, T, Hkv * G, Hkv, G, wl.k, wl.v)
    k, v, q = wlmod.make_k(w2, 50 + G), wlmod.make_v(w2, 50 + G), wlmod.make_q(w2, 50 + G)
    kb, vb, qb = wlmod.bf16_bits(k), wlmod.bf16_bits(v), wlmod.bf16_bits(q)
    records_k = torch.zeros((B, Hkv, t_cap, wl.k.record_bytes), dtype=torch.uint8, device=DEV)
    records_v = torch.zeros((B, Hkv, t_cap, wl.v.record_bytes), dtype=torch.uint8, device=DEV)
    mean_q = torch.zeros((B, Hkv, t_cap // 128, 128), dtype=torch.int8, device=DEV)
    mean_s = torch.zeros((B, Hkv, t_cap // 128), dtype=torch.int16, device=DEV)
    res_k = torch.full((B, Hkv, r_cap, 128), 30.0, dtype=torch.bfloat16, device=DEV)
    res_v = torch.full_like(res_k, -50.0)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    for b in range(B):
        n = comp[b]
        if n:
            dq.dq_encode_kv(gtk, kd[b:b + 1, :n], 0, t_cap, records_k[b:b + 1], mean_q[b:b + 1], mean_s[b:b + 1],
                            status)
            dq.dq_encode_kv(gtv, vd[b:b + 1, :n], 0, t_cap, records_v[b:b + 1], None, None, status)
        for i in range(res[b]):
            slot = (n + i) % r_cap
            res_k[b, :, slot] = kd[b, n + i]
            res_v[b, :, slot] = vd[b, n + i]
    seq = torch.tensor(comp, dtype=torch.int32, device=DEV)
    rl = torch.tensor(res, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_partial(gtk, gtv, qd, records_k, mean_q, mean_s, records_v, seq, ws, status=status)
    dq.dq_decode_attention_residual(qd, res_k, res_v, seq, rl, t_cap, ws)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    ref = _oracle(qb, kb, vb, comp, res, otk, otv, G)
    assert _rel_err(got, ref) < TOL
    assert _rel_err(_fused(dq, qd, res_k, res_v, seq, rl, t_cap, ws, got), ref) < TOL


@pytest.mark.parametrize("r_cap", [1, 3, 37, 130])
def test_residual_small_and_odd_rings(dq, r_cap):
    """Rings of any capacity up to 256: each of the four partial slots covers a
    quarter of the ring (some cover nothing when r_cap < 4), and the live
    tokens are the arc of res_lens[b] slots from seq_lens[b] mod r_cap."""
    wl = wlmod.workload("b1_t4k")
    otk = tables.build_tables(128, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(128, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, G, t_cap = 4, 1, 4, 256
    comp = [256, 128, 0, 128]
    res = [r_cap, max(0, r_cap - 1), min(r_cap, 2), r_cap // 2]
    T = max(c + r for c, r in zip(comp, res))
    w2 = wlmod.Workload("ring_small", B, T, Hkv * G, Hkv, 4, wl.k, wl.v)
    k, v, q = wlmod.make_k(w2, 31 + r_cap), wlmod.make_v(w2, 31 + r_cap), wlmod.make_q(w2, 31 + r_cap)
    kb, vb, qb = wlmod.bf16_bits(k), wlmod.bf16_bits(v), wlmod.bf16_bits(q)
    records_k = torch.zeros((B, Hkv, t_cap, wl.k.record_bytes), dtype=torch.uint8, device=DEV)
    records_v = torch.zeros((B, Hkv, t_cap, wl.v.record_bytes), dtype=torch.uint8, device=DEV)
    mean_q = torch.zeros((B, Hkv, t_cap // 128, 128), dtype=torch.int8, device=DEV)
    mean_s = torch.zeros((B, Hkv, t_cap // 128), dtype=torch.int16, device=DEV)
    # dead ring slots hold large values: a dead slot that leaked into the
    # softmax would show
    res_k = torch.full((B, Hkv, r_cap, 128), 30.0, dtype=torch.bfloat16, device=DEV)
    res_v = torch.full_like(res_k, -50.0)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    for b in range(B):
        n = comp[b]
        if n:
            dq.dq_encode_kv(gtk, kd[b:b + 1, :n], 0, t_cap, records_k[b:b + 1], mean_q[b:b + 1], mean_s[b:b + 1],
                            status)
            dq.dq_encode_kv(gtv, vd[b:b + 1, :n], 0, t_cap, records_v[b:b + 1], None, None, status)
        for i in range(res[b]):
            slot = (n + i) % r_cap
            res_k[b, :, slot] = kd[b, n + i]
            res_v[b, :, slot] = vd[b, n + i]
    seq = torch.tensor(comp, dtype=torch.int32, device=DEV)
    rl = torch.tensor(res, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_partial(gtk, gtv, qd, records_k, mean_q, mean_s, records_v, seq, ws, status=status)
    dq.dq_decode_attention_residual(qd, res_k, res_v, seq, rl, t_cap, ws)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    ref = _oracle(qb, kb, vb, comp, res, otk, otv, G)
    live = [b for b in range(B) if comp[b] + res[b] > 0]
    assert _rel_err(got[live], ref[live]) < TOL
    fused = _fused(dq, qd, res_k, res_v, seq, rl, t_cap, ws, got)
    assert _rel_err(fused[live], ref[live]) < TOL
    for b in range(B):
        if comp[b] + res[b] == 0:
            assert np.all(got[b] == 0.0)
            assert np.all(fused[b] == 0.0)


def test_streaming_cache_matches_oracle(dq):
    wl = wlmod.workload("b1_t4k")
    otk = tables.build_tables(128, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(128, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, G, prefill, steps = 2, 2, 4, 300, 300
    T = prefill + steps
    w2 = wlmod.Workload("stream", B, T, Hkv * G, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, 22)
    v = wlmod.make_v(w2, 22)
    kb, vb = wlmod.bf16_bits(k), wlmod.bf16_bits(v)
    kd, vd = k.to(DEV), v.to(DEV)
    cache = dq.StreamingKVCache(B, Hkv, Hkv * G, 1024, gtk, gtv)
    cache.prefill(kd[:, :prefill], vd[:, :prefill])
    checks = {prefill, prefill + 84, prefill + 85, prefill + 200, T}
    for t in range(prefill, T + 1):
        if t in checks:
            q = wlmod.make_q(w2, 1000 + t)
            out = cache.attend(q.to(DEV))
            torch.cuda.synchronize()
            assert int(cache.status.item()) == 0
            comp, res = cache.n_comp, cache.n_res
            assert comp + res == t and res >= min(t, 128) and comp % 128 == 0
            assert cache.seq_lens.tolist() == [comp] * B and cache.res_lens.tolist() == [res] * B
            ref = _oracle(wlmod.bf16_bits(q), kb, vb, [comp] * B, [res] * B, otk, otv, G)
            assert _rel_err(out.cpu().numpy().astype(np.float64), ref) < TOL
        if t < T:
            cache.append(kd[:, t].contiguous(), vd[:, t].contiguous())
    # the flushed windows are exactly the oracle's records of the same tokens
    n = cache.n_comp
    krec, mq, ms, _ = kv.encode_keys(kb[:, :n], otk)
    vrec, _ = kv.encode_values(vb[:, :n], otv)
    assert np.array_equal(cache.cache.k_records[:, :, :n].cpu().numpy(), krec)
    assert np.array_equal(cache.cache.v_records[:, :, :n].cpu().numpy(), vrec)
    assert np.array_equal(cache.cache.k_mean_q[:, :, :n // 128].cpu().numpy(), mq)


def test_ring_overflow_and_commit_flags(dq):
    B, Hkv, r_cap = 2, 1, 256
    res_k = torch.zeros((B, Hkv, r_cap, 128), dtype=torch.bfloat16, device=DEV)
    res_v = torch.zeros_like(res_k)
    seq = torch.zeros(B, dtype=torch.int32, device=DEV)
    rl = torch.tensor([r_cap, 3], dtype=torch.int32, device=DEV)      # first ring full
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    k1 = torch.ones((B, Hkv, 128), dtype=torch.bfloat16, device=DEV)
    dq.dq_residual_append(k1, k1, res_k, res_v, seq, rl, status)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_WINDOW
    assert rl.tolist() == [r_cap, 4]
    assert float(res_k[1, 0, 3, 0]) == 1.0 and float(res_k[0].abs().sum()) == 0.0
    status.zero_()
    dq.dq_residual_commit(seq, rl, 128, status)
    torch.cuda.synchronize()
    assert int(status.item()) & dq.DQ_STATUS_WINDOW          # the second ring holds only 4
    assert seq.tolist() == [128, 0] and rl.tolist() == [r_cap - 128, 4]


@pytest.mark.parametrize("G", [1, 3, 4, 8])
def test_fused_merge_many_chunks(dq, G):
    """The one-launch window + merge over many chunk partials: 128 and 78
    chunks of 256 tokens, so that a query head's rows arrive in many batches
    after the first and its maxima outnumber the lanes of a wavefront; 1, 3, 4
    and 8 query heads per KV head (at G < 8 some wavefronts only compute the
    window).  Checked against the two-call form (residual kernel, then the
    plain merge)."""
    wl = wlmod.workload("b1_t4k")
    gtk = dq.Tables(128, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    gtv = dq.Tables(128, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    B, Hkv, t_cap, r_cap = 2, 1, 32768, 256
    comp = [32768, 19968]
    res = [128, 37]
    T = max(c + r for c, r in zip(comp, res))
    w2 = wlmod.Workload("many_chunks", B, T, Hkv * G, Hkv, G, wl.k, wl.v)
    k, v, q = wlmod.make_k(w2, 70 + G), wlmod.make_v(w2, 70 + G), wlmod.make_q(w2, 70 + G)
    records_k = torch.zeros((B, Hkv, t_cap, wl.k.record_bytes), dtype=torch.uint8, device=DEV)
    records_v = torch.zeros((B, Hkv, t_cap, wl.v.record_bytes), dtype=torch.uint8, device=DEV)
    mean_q = torch.zeros((B, Hkv, t_cap // 128, 128), dtype=torch.int8, device=DEV)
    mean_s = torch.zeros((B, Hkv, t_cap // 128), dtype=torch.int16, device=DEV)
    res_k = torch.zeros((B, Hkv, r_cap, 128), dtype=torch.bfloat16, device=DEV)
    res_v = torch.zeros_like(res_k)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    for b in range(B):
        n = comp[b]
        dq.dq_encode_kv(gtk, kd[b:b + 1, :n], 0, t_cap, records_k[b:b + 1], mean_q[b:b + 1], mean_s[b:b + 1],
                        status)
        dq.dq_encode_kv(gtv, vd[b:b + 1, :n], 0, t_cap, records_v[b:b + 1], None, None, status)
        slots = [(n + i) % r_cap for i in range(res[b])]
        res_k[b, :, slots] = kd[b, n:n + res[b]].transpose(0, 1)
        res_v[b, :, slots] = vd[b, n:n + res[b]].transpose(0, 1)
    seq = torch.tensor(comp, dtype=torch.int32, device=DEV)
    rl = torch.tensor(res, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    qd = q.to(DEV)
    dq.dq_decode_attention_partial(gtk, gtv, qd, records_k, mean_q, mean_s, records_v, seq, ws, status=status)
    dq.dq_decode_attention_residual(qd, res_k, res_v, seq, rl, t_cap, ws)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    hdr = ws[:8].view(torch.int32).cpu().tolist()
    assert hdr[1] >= 64              # 128 chunks of 256 tokens on 256 CUs
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    _fused(dq, qd, res_k, res_v, seq, rl, t_cap, ws, got)
