"""Per-token streams at full size, in the launch configuration bench.py times
(--workload b16_t32k_tok: batch 16 x 32768 tokens, 32 query / 8 KV heads;
--workload b32_t32k_g8_tok: batch 32 x 32768 tokens, 64 query / 8 KV heads,
the second query-head slot group of the kernel): one 1024-value stream per
token and tensor (335 / 235-byte records in 336 / 240 byte slots, 8 / 6
levels, p 8), one prefill append per tensor, then the same partial + merge
calls.

The oracle cannot re-encode 524,288 tokens in seconds, so it checks what it
computes from the same seeded inputs:

* 128-token windows at scattered (sequence, window) positions, including the
  last window of the capacity: records (and their zero padding) and the key
  means of all 8 heads bit-exact;
* a decode step in the same launch configuration (same grid, chunking and
  wavefronts: those depend on the capacity, not on the lengths) where one
  sequence holds 2048 tokens: its 32 (64) query heads within 2e-3
  (row-normalized) of the oracle's fp64 attention over the oracle's own
  records;
* properties of the full-length launch: no status flag, finite outputs.
"""

import numpy as np
import pytest
import torch

import bench
import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables
from tokrec import from_tiles

pytestmark = pytest.mark.gpu

TOL = 2e-3
W = 128
SEED = 0          # bench.py's default seed


@pytest.fixture(scope="module", params=["b16_t32k_tok", "b32_t32k_g8_tok"])
def full(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = wlmod.workload(request.param)
    dev = torch.device("cuda")
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, dev)
    q, seq, out = bench.step_inputs(wl, SEED, dev)
    bench.decode_step(tk, tv, cache, q, seq, out)
    torch.cuda.synchronize()
    otk = tables.build_tables(wl.k.n, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes)
    otv = tables.build_tables(wl.v.n, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)
    return wl, cache, q, seq, out, otk, otv, tk, tv


def _inputs(wl, b, t0, t1):
    k = wlmod.make_k(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1]
    v = wlmod.make_v(wl, SEED * 1000 + b, device="cuda", batch=1)[:, t0:t1]
    return wlmod.bf16_bits(k), wlmod.bf16_bits(v)


def test_full_size_token_status_and_finite(full):
    wl, cache, q, seq, out, *_ = full
    assert int(cache.status.item()) == 0
    assert torch.isfinite(out).all()


@pytest.mark.parametrize("b,w", [(0, 0), (7, 128), (15, 255)])
def test_full_size_token_windows_bit_exact(full, b, w):
    wl, cache, q, seq, out, otk, otv, *_ = full
    t0 = w * W
    k, v = _inputs(wl, b, t0, t0 + W)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(k, otk)
    vrec, _ = kv.encode_values_tokenwise(v, otv)
    gk = from_tiles(cache.k_records[b:b + 1, t0 // 64:(t0 + W) // 64].cpu().numpy())[0]
    gv = from_tiles(cache.v_records[b:b + 1, t0 // 64:(t0 + W) // 64].cpu().numpy())[0]
    assert np.array_equal(gk[:, :otk.record_bytes], krec[0]) and not gk[:, otk.record_bytes:].any()
    assert np.array_equal(gv[:, :otv.record_bytes], vrec[0]) and not gv[:, otv.record_bytes:].any()
    assert np.array_equal(cache.k_mean_q[b, :, w].cpu().numpy(), mq[0, :, 0])
    assert np.array_equal(cache.k_mean_scale[b, :, w].cpu().numpy().view(np.uint16), ms[0, :, 0].view(np.uint16))


def test_full_size_token_attention_short_sequence(full):
    wl, cache, q, seq, out, otk, otv, tk, tv = full
    b, T = 11, 2048
    lens = seq.clone()
    lens[b] = T
    out2 = torch.empty_like(out)
    bench.decode_step(tk, tv, cache, q, lens, out2)
    torch.cuda.synchronize()
    assert int(cache.status.item()) == 0
    # the other sequences are untouched by the change of length
    keep = [i for i in range(wl.batch) if i != b]
    assert torch.equal(out2[keep], out[keep])
    k, v = _inputs(wl, b, 0, T)
    krec, mq, ms, _ = kv.encode_keys_tokenwise(k, otk)
    vrec, _ = kv.encode_values_tokenwise(v, otv)
    H = wl.kv_heads
    ksym, ks, ko, _ = kv.decode_records(krec, otk, wl.k.n)
    vsym, vs, vo, _ = kv.decode_records(vrec, otv, wl.v.n)
    kh, ksh, koh = kv.tokenwise_as_heads(ksym, ks, ko, H)
    vh, vsh, voh = kv.tokenwise_as_heads(vsym, vs, vo, H)
    qb = wlmod.bf16_bits(q[b:b + 1])
    ref = attention.attention_folded(kv.bf16_to_f64(qb), kh, ksh, koh, kmean.dequantize_mean(mq, ms),
                                     vh, vsh, voh, [T], wl.gqa, 1 / np.sqrt(wl.head_dim))
    got = out2[b:b + 1].cpu().numpy().astype(np.float64)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got - ref) / scale)) < TOL
