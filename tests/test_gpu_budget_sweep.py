"""The long-context bit-budget sweep at its full size, in the launch
configuration bench.py times (--workload b1_t128k --bpe B [--variant literal]):
batch 1 x 131072 tokens x 8 KV heads, 32 query heads, records of 32 / 36 / 48
/ 64 bytes (2.0 / 2.26 / 3.0 / 4.0 bits per element) with the stated level
counts 16 / 16 / 32 / 64 ("literal", alpha raised until the count fits) and
with the paper's level counts at alpha = 1.4 ("paper").  The cache is filled
by one encode call per tensor and decoded by the same partial + merge calls.

The oracle cannot re-encode 2 M streams per case in seconds, so it checks what
it computes from the same seeded inputs:

* 128-token windows (the first and the last of the capacity) of one KV head:
  records and key means bit-exact;
* a decode step in the same launch configuration (grid and chunking depend on
  the capacity, not on the lengths) where the sequence holds 1536 tokens: one
  KV head's 4 query heads within 2e-3 (row-normalized) of the oracle's fp64
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
SWEEP = [(bpe, variant) for bpe in (2.0, 2.26, 3.0, 4.0) for variant in ("paper", "literal")]


@pytest.fixture(scope="module", params=SWEEP, ids=lambda p: f"{p[0]}-{p[1]}")
def sweep(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bpe, variant = request.param
    wl = wlmod.workload("b1_t128k", variant, bpe)
    dev = torch.device("cuda")
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, dev)
    q, seq, out = bench.step_inputs(wl, SEED, dev)
    bench.decode_step(tk, tv, cache, q, seq, out)
    short = seq.clone()
    short[0] = T_SHORT
    out_short = torch.empty_like(out)
    bench.decode_step(tk, tv, cache, q, short, out_short)
    torch.cuda.synchronize()
    otk = tables.build_tables(wl.head_dim, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(wl.head_dim, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    yield wl, cache, q, out, out_short, otk, otv
    del cache
    torch.cuda.empty_cache()


def _inputs(wl, h, t0, t1):
    k = wlmod.make_k(wl, SEED * 1000, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    v = wlmod.make_v(wl, SEED * 1000, device="cuda", batch=1)[:, t0:t1, h:h + 1]
    return wlmod.bf16_bits(k), wlmod.bf16_bits(v)


def test_sweep_status_and_finite(sweep):
    wl, cache, q, out, out_short, otk, otv = sweep
    assert otk.record_bytes == wl.k.record_bytes and otk.M == wl.k.levels
    assert int(cache.status.item()) == 0
    assert torch.isfinite(out).all() and torch.isfinite(out_short).all()


@pytest.mark.parametrize("h,w", [(2, 0), (6, 131072 // W - 1)])
def test_sweep_windows_bit_exact(sweep, h, w):
    wl, cache, _, _, _, otk, otv = sweep
    t0, t1 = w * W, (w + 1) * W
    k, v = _inputs(wl, h, t0, t1)
    krec, mq, ms, _ = kv.encode_keys(k, otk)
    vrec, _ = kv.encode_values(v, otv)
    assert np.array_equal(cache.k_records[0, h, t0:t1].cpu().numpy(), krec[0, 0])
    assert np.array_equal(cache.v_records[0, h, t0:t1].cpu().numpy(), vrec[0, 0])
    assert np.array_equal(cache.k_mean_q[0, h, w].cpu().numpy(), mq[0, 0, 0])
    assert cache.k_mean_scale[0, h, w].item() & 0xFFFF == int(ms[0, 0, 0:1].view(np.uint16)[0])


def test_sweep_short_sequence_attention(sweep):
    wl, cache, q, _, out_short, otk, otv = sweep
    h, G = 5, wl.gqa
    k, v = _inputs(wl, h, 0, T_SHORT)
    krec, mq, ms, ksym = kv.encode_keys(k, otk)
    vrec, vsym = kv.encode_values(v, otv)
    _, ks, ko, _ = kv.decode_records(krec, otk, wl.head_dim)
    _, vs, vo, _ = kv.decode_records(vrec, otv, wl.head_dim)
    qb = wlmod.bf16_bits(q[0:1, h * G:(h + 1) * G])
    ref = attention.attention_folded(kv.bf16_to_f64(qb), ksym, ks, ko, kmean.dequantize_mean(mq, ms),
                                     vsym, vs, vo, [T_SHORT], G, 1 / np.sqrt(wl.head_dim))
    got = out_short[0:1, h * G:(h + 1) * G].cpu().numpy().astype(np.float64)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got - ref) / scale)) < TOL
