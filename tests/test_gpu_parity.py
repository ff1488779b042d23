"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bars: records, symbols and key means bit-exact; attention within 2e-3 of the
oracle's fp64 attention over the same records, measured as
max |y - y_ref| / max_j |y_ref[b, i, :]| (row-normalized).
Every expected value comes from the oracle on the same seeded inputs; oracle
records are uploaded to the GPU for the attention checks.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kmean, kv, rans, tables

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


DEV = "cuda"


def _tabs(dq, coding, n=128):
    return (dq.Tables(n, coding.levels, coding.precision, coding.record_bytes, coding.alpha),
            tables.build_tables(n, coding.levels, coding.precision, coding.alpha, coding.record_bytes))


def _rel_err(got, ref):
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    return float(np.max(np.abs(got - ref) / np.maximum(scale, 1e-30)))


def _oracle_attention(q_bits, krec, mq, ms, vrec, otk, otv, lens, G):
    ksym, ks, ko, okk = kv.decode_records(krec, otk, 128)
    vsym, vs, vo, okv = kv.decode_records(vrec, otv, 128)
    assert okk.all() and okv.all()
    return attention.attention_folded(kv.bf16_to_f64(q_bits), ksym, ks, ko, kmean.dequantize_mean(mq, ms),
                                      vsym, vs, vo, lens, G, 1 / np.sqrt(128))


# ------------------------------------------------------------------ symbols

@pytest.mark.parametrize("variant", ["paper", "literal"])
def test_decode_symbols_bit_exact(dq, variant):
    wl = wlmod.workload("b1_t4k", variant)
    gt, ot = _tabs(dq, wl.k)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 1, batch=1, context=384))
    krec, _, _, ksym = kv.encode_keys(k, ot)
    rec = torch.from_numpy(krec).to(DEV)
    S = krec.size // ot.record_bytes
    sym = torch.empty((S, 128), dtype=torch.uint8, device=DEV)
    hdr = torch.empty((S, 2), dtype=torch.int16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_decode_symbols(gt, rec, sym, hdr, status)
    torch.cuda.synchronize()
    assert np.array_equal(sym.cpu().numpy().reshape(ksym.shape), ksym)
    h = hdr.cpu().numpy().view(np.uint16)
    r = krec.reshape(-1, ot.record_bytes).astype(np.uint16)
    assert np.array_equal(h[:, 0], r[:, 0] | (r[:, 1] << 8))
    assert np.array_equal(h[:, 1], r[:, 2] | (r[:, 3] << 8))
    assert int(status.item()) == 0


def test_decode_symbols_malformed_records(dq):
    """Random bytes: both decoders stop at the record end and agree symbol for
    symbol; the GPU raises the corrupt-record flag."""
    wl = wlmod.workload("b1_t4k")
    gt, ot = _tabs(dq, wl.v)
    rng = np.random.default_rng(3)
    recs = rng.integers(0, 256, size=(500, ot.record_bytes), dtype=np.uint8)
    recs[:5] = 0
    ref, x, _ = rans.decode(recs, ot, 128)
    sym = torch.empty((500, 128), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_decode_symbols(gt, torch.from_numpy(recs).to(DEV), sym, None, status)
    torch.cuda.synchronize()
    assert np.array_equal(sym.cpu().numpy(), ref)
    assert (int(status.item()) & dq.DQ_STATUS_CORRUPT) and np.any(x != rans.RANS_L)


# ------------------------------------------------------------------- encode

def _gpu_encode(dq, gt, x_bf16, t0, t_cap, keys, records=None, mq=None, ms=None):
    B, T, H, d = x_bf16.shape
    if records is None:
        records = torch.zeros((B, H, t_cap, gt.record_bytes), dtype=torch.uint8, device=DEV)
    if keys and mq is None:
        mq = torch.zeros((B, H, t_cap // 128, d), dtype=torch.int8, device=DEV)
        ms = torch.zeros((B, H, t_cap // 128), dtype=torch.int16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_encode_kv(gt, x_bf16, t0, t_cap, records, mq if keys else None, ms if keys else None, status)
    torch.cuda.synchronize()
    return records, mq, ms, int(status.item())


@pytest.mark.parametrize("variant", ["paper", "literal"])
def test_encode_keys_bit_exact(dq, variant):
    wl = wlmod.workload("b1_t4k", variant)
    gt, ot = _tabs(dq, wl.k)
    k = wlmod.make_k(wl, 2, batch=2, context=256)
    rec, mq, ms, st = _gpu_encode(dq, gt, k.to(DEV), 0, 256, True)
    krec, omq, oms, _ = kv.encode_keys(wlmod.bf16_bits(k), ot)
    assert st == 0
    assert np.array_equal(mq.cpu().numpy(), omq)
    assert np.array_equal(ms.cpu().numpy().view(np.uint16), oms.view(np.uint16))
    got = rec.cpu().numpy()
    bad = np.argwhere(np.any(got != krec, axis=-1))
    assert bad.size == 0, f"{len(bad)} records differ, first {bad[:3].tolist()}"


@pytest.mark.parametrize("variant", ["paper", "literal"])
def test_encode_values_bit_exact(dq, variant):
    wl = wlmod.workload("b1_t4k", variant)
    gt, ot = _tabs(dq, wl.v)
    v = wlmod.make_v(wl, 4, batch=2, context=256)
    rec, _, _, st = _gpu_encode(dq, gt, v.to(DEV), 0, 256, False)
    vrec, _ = kv.encode_values(wlmod.bf16_bits(v), ot)
    assert st == 0
    assert np.array_equal(rec.cpu().numpy(), vrec)


def test_encode_appends_at_offsets_and_ragged_tail(dq):
    """Values appended in pieces of 100, 1 and 27 tokens (ragged workgroups)
    equal a one-shot oracle encode; untouched slots stay zero."""
    wl = wlmod.workload("b1_t4k")
    gt, ot = _tabs(dq, wl.v)
    v = wlmod.make_v(wl, 5, batch=1, context=128)
    rec = torch.zeros((1, 8, 256, gt.record_bytes), dtype=torch.uint8, device=DEV)
    vd = v.to(DEV)
    for a, b in ((0, 100), (100, 101), (101, 128)):
        _gpu_encode(dq, gt, vd[:, a:b], a, 256, False, records=rec)
    vrec, _ = kv.encode_values(wlmod.bf16_bits(v), ot)
    got = rec.cpu().numpy()
    assert np.array_equal(got[:, :, :128], vrec)
    assert not got[:, :, 128:].any()


def test_encode_key_windows_at_offset(dq):
    wl = wlmod.workload("b1_t4k")
    gt, ot = _tabs(dq, wl.k)
    k = wlmod.make_k(wl, 6, batch=1, context=256)
    rec, mq, ms, _ = _gpu_encode(dq, gt, k[:, :128].to(DEV), 0, 384, True)
    rec, mq, ms, _ = _gpu_encode(dq, gt, k[:, 128:].to(DEV), 128, 384, True, records=rec, mq=mq, ms=ms)
    krec, omq, oms, _ = kv.encode_keys(wlmod.bf16_bits(k), ot)
    assert np.array_equal(rec.cpu().numpy()[:, :, :256], krec)
    assert np.array_equal(mq.cpu().numpy()[:, :, :2], omq)


def test_encode_strided_input(dq):
    """kv may be a strided view (e.g. one slice of a fused QKV projection)."""
    wl = wlmod.workload("b1_t4k")
    gt, ot = _tabs(dq, wl.v)
    v = wlmod.make_v(wl, 7, batch=2, context=128)
    big = torch.zeros((2, 128, 8, 3, 128), dtype=torch.bfloat16)
    big[:, :, :, 1] = v
    view = big.to(DEV)[:, :, :, 1]
    assert not view.is_contiguous()
    rec, _, _, _ = _gpu_encode(dq, gt, view, 0, 128, False)
    vrec, _ = kv.encode_values(wlmod.bf16_bits(v), ot)
    assert np.array_equal(rec.cpu().numpy(), vrec)


def test_encode_wide_gqa_asymmetric_budgets(dq):
    """Keys at 3.0 bits/elem (48 B), values at 2.0 (32 B), 8 outlier channels."""
    for variant in ("paper", "literal"):
        wl = wlmod.workload("b32_t32k_g8", variant)
        for coding, keys, seed in ((wl.k, True, 8), (wl.v, False, 9)):
            gt, ot = _tabs(dq, coding)
            x = (wlmod.make_k if keys else wlmod.make_v)(wl, seed, batch=1, context=128)
            rec, mq, ms, st = _gpu_encode(dq, gt, x.to(DEV), 0, 128, keys)
            if keys:
                ref = kv.encode_keys(wlmod.bf16_bits(x), ot)[0]
            else:
                ref = kv.encode_values(wlmod.bf16_bits(x), ot)[0]
            assert st == 0 and np.array_equal(rec.cpu().numpy(), ref), (variant, keys)


@pytest.mark.parametrize("n", [64, 256])
def test_encode_other_head_dims(dq, n):
    """The encoder's wavefront layout for 1 and 4 values per lane."""
    C = {64: 24, 256: 72}[n]
    gt = dq.Tables(n, 6, 12, C, 1.4)
    ot = tables.build_tables(n, 6, 12, 1.4, C)
    g = torch.Generator().manual_seed(n)
    x = (torch.randn((1, 128, 2, n), generator=g) * 3 + 1).to(torch.bfloat16)
    rec, mq, ms, _ = _gpu_encode(dq, gt, x.to(DEV), 0, 128, True)
    krec, omq, oms, _ = kv.encode_keys(wlmod.bf16_bits(x), ot)
    assert np.array_equal(mq.cpu().numpy(), omq)
    assert np.array_equal(rec.cpu().numpy(), krec)


def test_encode_flags_non_finite_input(dq):
    wl = wlmod.workload("b1_t4k")
    gt, _ = _tabs(dq, wl.v)
    v = wlmod.make_v(wl, 0, batch=1, context=64).to(DEV)
    v[0, 3, 2, 5] = float("inf")
    _, _, _, st = _gpu_encode(dq, gt, v, 0, 128, False)
    assert st & dq.DQ_STATUS_RANGE


def test_encode_deterministic(dq):
    wl = wlmod.workload("b1_t4k")
    gt, _ = _tabs(dq, wl.k)
    k = wlmod.make_k(wl, 3, batch=2, context=512).to(DEV)
    a = _gpu_encode(dq, gt, k, 0, 512, True)[0].cpu()
    b = _gpu_encode(dq, gt, k, 0, 512, True)[0].cpu()
    assert torch.equal(a, b)


# ---------------------------------------------------------------- attention

def _upload_cache(dq, wl, krec, mq, ms, vrec):
    return (torch.from_numpy(krec).to(DEV), torch.from_numpy(mq).to(DEV),
            torch.from_numpy(ms.view(np.int16)).to(DEV), torch.from_numpy(vrec).to(DEV))


def _pad_capacity(kr, mq, ms, vr, t_cap):
    """The same cache in buffers of capacity t_cap (zero rows past the old
    one).  The chunk plan follows the capacity, not the lengths: on a 256-CU
    device a capacity of 32 x 1024 tokens per (sequence, KV head) pair gives
    1024-token chunks (16 tiles), which one wavefront per tile decodes with
    both chains (the split form takes chunks of at most half as many tiles
    as a workgroup has wavefronts)."""
    def pad(x, n):
        shape = list(x.shape)
        shape[2] = n
        y = torch.zeros(shape, dtype=x.dtype, device=x.device)
        y[:, :, :x.shape[2]] = x
        return y
    return pad(kr, t_cap), pad(mq, t_cap // 128), pad(ms, t_cap // 128), pad(vr, t_cap)


JOINT_CAP = 32768     # b1_t4k-like batches: 1024-token chunks, the two-chain form


def _gpu_attention(dq, gtk, gtv, q, kr, mq, ms, vr, lens, Hq, t_cap=None):
    B = q.shape[0]
    if t_cap is not None:
        kr, mq, ms, vr = _pad_capacity(kr, mq, ms, vr, t_cap)
    Hkv, t_cap = kr.shape[1], kr.shape[2]
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hq, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    dq.dq_decode_attention(gtk, gtv, q.to(DEV), kr, mq, ms, vr, seq, out, ws, status=status)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), int(status.item())


@pytest.mark.parametrize("variant,cap", [("paper", None), ("literal", None), ("paper", JOINT_CAP)])
def test_attention_small_workload(dq, variant, cap):
    """Full b1_t4k workload: batch 1, 32/8 heads, 4096 tokens (keys and values
    in separate wavefronts; in larger buffers, with both chains in one)."""
    wl = wlmod.workload("b1_t4k", variant)
    gtk, otk = _tabs(dq, wl.k)
    gtv, otv = _tabs(dq, wl.v)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 0))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 0))
    q = wlmod.make_q(wl, 0)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    ref = _oracle_attention(wlmod.bf16_bits(q), krec, mq, ms, vrec, otk, otv, [4096], wl.gqa)
    got, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl, krec, mq, ms, vrec), [4096], wl.q_heads,
                             t_cap=cap)
    assert st == 0
    assert _rel_err(got, ref) < TOL


@pytest.mark.parametrize("cap", [None, 4096])
def test_attention_ragged_lengths(dq, cap):
    """Lengths 0, 1, 63, 64, 65, 127, 128, 129, 300, 512 in one batch; in
    buffers of 512 tokens (split form) and of 4096 (1024-token chunks, both
    chains in one wavefront)."""
    wl = wlmod.workload("b1_t4k")
    gtk, otk = _tabs(dq, wl.k)
    gtv, otv = _tabs(dq, wl.v)
    lens = [0, 1, 63, 64, 65, 127, 128, 129, 300, 512]
    B, T = len(lens), 512
    k = wlmod.bf16_bits(wlmod.make_k(wl, 11, batch=B, context=T))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 11, batch=B, context=T))
    q = wlmod.make_q(wl, 11, batch=B)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    got, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl, krec, mq, ms, vrec), lens, wl.q_heads,
                             t_cap=cap)
    assert st == 0
    assert np.all(got[0] == 0.0)
    ref = _oracle_attention(wlmod.bf16_bits(q)[1:], krec[1:], mq[1:], ms[1:], vrec[1:], otk, otv, lens[1:], wl.gqa)
    assert _rel_err(got[1:], ref) < TOL


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_attention_gqa_groups(dq, G):
    wl = wlmod.workload("b32_t32k_g8")     # keys 48 B / values 32 B
    gtk, otk = _tabs(dq, wl.k)
    gtv, otv = _tabs(dq, wl.v)
    B, T, Hkv = 2, 1024, 8 // G if G == 8 else 4
    Hq = Hkv * G
    wl2 = wlmod.Workload("g", B, T, Hq, Hkv, 8, wl.k, wl.v)
    k = wlmod.bf16_bits(wlmod.make_k(wl2, 12))
    v = wlmod.bf16_bits(wlmod.make_v(wl2, 12))
    q = wlmod.make_q(wl2, 12)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    lens = [1024, 700]
    ref = _oracle_attention(wlmod.bf16_bits(q), krec, mq, ms, vrec, otk, otv, lens, G)
    got, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl2, krec, mq, ms, vrec), lens, Hq)
    assert st == 0
    assert _rel_err(got, ref) < TOL


@pytest.mark.parametrize("C,G,cap", [(32, 4, None), (36, 8, None), (48, 4, None), (64, 4, None), (64, 8, None),
                                     (36, 1, None), (36, 2, None),
                                     (32, 4, 65536), (48, 4, 65536), (64, 4, 65536), (36, 2, 65536)])
def test_attention_record_lengths(dq, C, G, cap):
    """Equal key/value record lengths of the 2.0 / 2.25 / 3.0 / 4.0 bits-per-
    element budgets (paper level counts), 1, 2, 4 and 8 query heads per KV
    head; up to 4 also in buffers of 65536 tokens (2048-token chunks, both
    chains in one wavefront)."""
    coding = wlmod.Coding(levels=wlmod.PAPER_LEVELS[C], record_bytes=C, alpha=1.4)
    gtk, otk = _tabs(dq, coding)
    B, T, Hkv = 2, 1536, 2
    wl = wlmod.Workload("r", B, T, Hkv * G, Hkv, 4, coding, coding)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 15))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 15))
    q = wlmod.make_q(wl, 15)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otk)
    lens = [1536, 1000]
    ref = _oracle_attention(wlmod.bf16_bits(q), krec, mq, ms, vrec, otk, otk, lens, G)
    got, st = _gpu_attention(dq, gtk, gtk, q, *_upload_cache(dq, wl, krec, mq, ms, vrec), lens, Hkv * G,
                             t_cap=cap)
    assert st == 0
    assert _rel_err(got, ref) < TOL


@pytest.mark.parametrize("cap", [None, JOINT_CAP])
def test_attention_flags_corrupt_record(dq, cap):
    wl = wlmod.workload("b1_t4k")
    gtk, otk = _tabs(dq, wl.k)
    gtv, otv = _tabs(dq, wl.v)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 13, batch=1, context=256))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 13, batch=1, context=256))
    q = wlmod.make_q(wl, 13, batch=1)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    vrec[0, 3, 17, 5] ^= 0x40
    _, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl, krec, mq, ms, vrec), [256], wl.q_heads,
                           t_cap=cap)
    assert st & dq.DQ_STATUS_CORRUPT
    # the same in a key record
    vrec[0, 3, 17, 5] ^= 0x40
    krec1 = krec.copy()
    krec1[0, 5, 40, 5] ^= 0x40
    _, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl, krec1, mq, ms, vrec), [256], wl.q_heads,
                           t_cap=cap)
    assert st & dq.DQ_STATUS_CORRUPT
    # a corrupt record past the sequence length is never read
    krec2 = krec.copy()
    krec2[0, 0, 200, 6] ^= 0x40
    _, st = _gpu_attention(dq, gtk, gtv, q, *_upload_cache(dq, wl, krec2, mq, ms, vrec), [128], wl.q_heads,
                           t_cap=cap)
    assert st == 0


def test_attention_deterministic(dq):
    wl = wlmod.workload("b1_t4k")
    gtk, otk = _tabs(dq, wl.k)
    gtv, otv = _tabs(dq, wl.v)
    k = wlmod.bf16_bits(wlmod.make_k(wl, 14, batch=1, context=512))
    v = wlmod.bf16_bits(wlmod.make_v(wl, 14, batch=1, context=512))
    q = wlmod.make_q(wl, 14, batch=1)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    cache = _upload_cache(dq, wl, krec, mq, ms, vrec)
    a, _ = _gpu_attention(dq, gtk, gtv, q, *cache, [512], wl.q_heads)
    b, _ = _gpu_attention(dq, gtk, gtv, q, *cache, [512], wl.q_heads)
    assert np.array_equal(a, b)
