"""Parity at the full sizes of the high-batch and wide-group workloads, in
the launch configuration bench.py times: b64_t8k (batch 64 x 8192 tokens x 8
KV heads, 36-byte records) and b32_t32k_g8 (batch 32 x 32768 tokens, 64 query
/ 8 KV heads, 48-byte keys and 32-byte values).  The cache is filled as the
benchmark fills it and one decode step runs through the same partial + merge
calls.  The oracle checks what it computes from the same seeded inputs:

* 128-token windows at scattered (sequence, KV head, window) positions:
  records and key means bit-exact;
* a decode step in the same launch configuration (grid and chunking depend on
  the capacity, not on the lengths) where one sequence holds 1536 tokens: that
  KV head's G query heads within 2e-3 (row-normalized) of the oracle's fp64
  attention over the oracle's own records;
* properties of the full-length launch: no status flag, finite outputs.
"""

import numpy as np
import pytest
import torch

import bench
import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables

pytestmark = pytest.mark.gpu

TOL = 2e-3
W = 128
SEED = 0          # bench.py's default seed
T_SHORT = 1536
# (workload, sequence and KV head of the short-sequence check, sampled windows)
CASES = {
    "b64_t8k": (41, 6, [(0, 0, 0), (17, 3, 63), (63, 7, 31)]),
    "b32_t32k_g8": (19, 2, [(0, 1, 0), (12, 4, 255), (31, 7, 130)]),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def full(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = wlmod.workload(request.param, "paper")
    dev = torch.device("cuda")
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, dev)
    q, seq, out = bench.step_inputs(wl, SEED, dev)
    bench.decode_step(tk, tv, cache, q, seq, out)
    sb, sh, _ = CASES[request.param]
    short = seq.clone()
    short[sb] = T_SHORT
    out_short = torch.empty_like(out)
    bench.decode_step(tk, tv, cache, q, short, out_short)
    torch.cuda.synchronize()
    otk = tables.build_tables(wl.head_dim, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(wl.head_dim, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    yield request.param, wl, cache, q, out, out_short, otk, otv
    del cache
    torch.cuda.empty_cache()


def _inputs(wl, b, h, t0, t1):
    """bf16 bits of K and V for sequence b, KV head h, tokens [t0, t1), from
    the same device generator the cache was filled from."""
    k = wlmod.make_k(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    v = wlmod.make_v(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    return wlmod.bf16_bits(k), wlmod.bf16_bits(v)


def test_full_size_status_and_finite(full):
    _, wl, cache, q, out, out_short, _, _ = full
    assert int(cache.status.item()) == 0
    assert torch.isfinite(out).all() and torch.isfinite(out_short).all()


def test_full_size_sampled_windows(full):
    name, wl, cache, _, _, _, otk, otv = full
    for b, h, w in CASES[name][2]:
        t0, t1 = w * W, (w + 1) * W
        k, v = _inputs(wl, b, h, t0, t1)
        krec, mq, ms, _ = kv.encode_keys(k, otk)
        vrec, _ = kv.encode_values(v, otv)
        assert np.array_equal(cache.k_records[b, h, t0:t1].cpu().numpy(), krec[0, 0]), (b, h, w)
        assert np.array_equal(cache.v_records[b, h, t0:t1].cpu().numpy(), vrec[0, 0]), (b, h, w)
        assert np.array_equal(cache.k_mean_q[b, h, w].cpu().numpy(), mq[0, 0, 0]), (b, h, w)
        assert cache.k_mean_scale[b, h, w].item() & 0xFFFF == int(ms[0, 0, 0:1].view(np.uint16)[0])


def test_full_size_short_sequence_attention(full):
    name, wl, cache, q, _, out_short, otk, otv = full
    b, h, _ = CASES[name]
    G = wl.gqa
    k, v = _inputs(wl, b, h, 0, T_SHORT)
    krec, mq, ms, ksym = kv.encode_keys(k, otk)
    vrec, vsym = kv.encode_values(v, otv)
    _, ks, ko, _ = kv.decode_records(krec, otk, wl.head_dim)
    _, vs, vo, _ = kv.decode_records(vrec, otv, wl.head_dim)
    qb = wlmod.bf16_bits(q[b:b + 1, h * G:(h + 1) * G])
    ref = attention.attention_folded(kv.bf16_to_f64(qb), ksym, ks, ko, kmean.dequantize_mean(mq, ms),
                                     vsym, vs, vo, [T_SHORT], G, 1 / np.sqrt(wl.head_dim))
    got = out_short[b:b + 1, h * G:(h + 1) * G].cpu().numpy().astype(np.float64)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got - ref) / scale)) < TOL
