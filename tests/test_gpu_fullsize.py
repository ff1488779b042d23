"""Parity at the full b16_t32k size, in the launch configuration bench.py times.

The cache is filled exactly as the benchmark fills it (batch 16 x 32768
tokens x 8 KV heads, 36-byte records, one encode call per sequence) and one
decode step runs through the same partial + merge calls.  The oracle cannot
redo all 4.2 M streams in seconds, so it checks samples it computes one by one
from the same seeded inputs:

* one whole (sequence, KV head) slice: all 32768 key and value records and the
  256 key means bit-exact, and the attention output of its 4 query heads
  within 2e-3 (row-normalized) of the oracle's fp64 attention over the
  oracle's own records;
* 128-token windows at scattered (sequence, KV head, window) positions:
  records and key means bit-exact;
* properties of the whole launch: no status flag, finite outputs.
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


@pytest.fixture(scope="module")
def full():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = wlmod.workload("b16_t32k", "paper")
    dev = torch.device("cuda")
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, dev)
    q, seq, out = bench.step_inputs(wl, SEED, dev)
    bench.decode_step(tk, tv, cache, q, seq, out)
    torch.cuda.synchronize()
    otk = tables.build_tables(wl.head_dim, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(wl.head_dim, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    return wl, cache, q, out, otk, otv


def _inputs(wl, b, h, t0, t1):
    """bf16 bits of K and V for sequence b, KV head h, tokens [t0, t1), from
    the same device generator the cache was filled from."""
    k = wlmod.make_k(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    v = wlmod.make_v(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    return wlmod.bf16_bits(k), wlmod.bf16_bits(v)


def test_full_size_status_and_finite(full):
    wl, cache, q, out, _, _ = full
    assert int(cache.status.item()) == 0
    assert torch.isfinite(out).all()


def test_full_size_slice_records_and_attention(full):
    wl, cache, q, out, otk, otv = full
    b, h, G, T = 15, 7, wl.gqa, wl.context
    k, v = _inputs(wl, b, h, 0, T)
    krec, mq, ms, ksym = kv.encode_keys(k, otk)
    vrec, vsym = kv.encode_values(v, otv)
    assert np.array_equal(cache.k_records[b, h].cpu().numpy(), krec[0, 0])
    assert np.array_equal(cache.v_records[b, h].cpu().numpy(), vrec[0, 0])
    assert np.array_equal(cache.k_mean_q[b, h].cpu().numpy(), mq[0, 0])
    assert np.array_equal(cache.k_mean_scale[b, h].cpu().numpy().view(np.uint16), ms[0, 0].view(np.uint16))

    _, ks, ko, _ = kv.decode_records(krec, otk, wl.head_dim)
    _, vs, vo, _ = kv.decode_records(vrec, otv, wl.head_dim)
    qb = wlmod.bf16_bits(q[b:b + 1, h * G:(h + 1) * G])
    ref = attention.attention_folded(kv.bf16_to_f64(qb), ksym, ks, ko, kmean.dequantize_mean(mq, ms),
                                     vsym, vs, vo, [T], G, 1 / np.sqrt(wl.head_dim))
    got = out[b:b + 1, h * G:(h + 1) * G].cpu().numpy().astype(np.float64)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got - ref) / scale)) < TOL


@pytest.mark.parametrize("b,h,w", [(0, 0, 0), (0, 3, 255), (4, 1, 17), (9, 5, 128), (12, 2, 200), (15, 7, 63)])
def test_full_size_sampled_windows(full, b, h, w):
    wl, cache, _, _, otk, otv = full
    t0, t1 = w * W, (w + 1) * W
    k, v = _inputs(wl, b, h, t0, t1)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    assert np.array_equal(cache.k_records[b, h, t0:t1].cpu().numpy(), krec[0, 0])
    assert np.array_equal(cache.v_records[b, h, t0:t1].cpu().numpy(), vrec[0, 0])
    assert np.array_equal(cache.k_mean_q[b, h, w].cpu().numpy(), mq[0, 0, 0])
    assert cache.k_mean_scale[b, h, w].item() & 0xFFFF == int(ms[0, 0, 0:1].view(np.uint16)[0])
