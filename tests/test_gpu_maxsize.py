"""Decode attention at the largest capacity the tests allocate: batch 4 x
2^21 tokens x 8 KV heads (32 query heads), 36-byte key and value records:
4.8 GB of records whose byte offsets pass 2^31, 128 split-K chunks per
sequence.

The expected output is fixed by construction so that the oracle can compute
it from 128 tokens: the key and value records repeat one 128-token unit that
the oracle encoded (one key-mean window, whose mean then stands in every
window), so the logits repeat with period 128 and, over any length that is a
multiple of 128, the softmax gives each period the same weights: the output
equals the oracle's attention over the unit alone.  Lengths 2^21,
2^21 - 128 x 4099, 2^20 and 128 run in one batch, each sequence with its own
query; each output row must be within 2e-3 (row-normalized) of the oracle's.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kmean, kv, tables

pytestmark = pytest.mark.gpu

TOL = 2e-3
DEV = "cuda"
B, HKV, G, D = 4, 8, 4, 128
T_CAP = 1 << 21
W = 128


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


def test_max_capacity_periodic_cache(dq):
    wl = wlmod.workload("b16_t32k")
    c = wl.k
    C = c.record_bytes
    gt = dq.Tables(D, c.levels, c.precision, C, c.alpha)
    ot = tables.build_tables(D, c.levels, c.precision, c.alpha, C)

    unit = wl.with_context(W, batch=1)
    krec, mq, ms, _ = kv.encode_keys(wlmod.bf16_bits(wlmod.make_k(unit, 21)), ot)   # [1, H, 128, C]
    vrec, _ = kv.encode_values(wlmod.bf16_bits(wlmod.make_v(unit, 21)), ot)
    q = wlmod.make_q(wl, 22, batch=B)                                              # [B, Hq, d]

    # the cache: the 128-token unit of key and value records repeated along
    # the context, the unit's key mean in every window
    def periodic(rec):
        u = torch.from_numpy(np.ascontiguousarray(rec[0])).to(DEV)                # [H, 128, C]
        return u[None, :, None].expand(B, HKV, T_CAP // W, W, C).reshape(B, HKV, T_CAP, C)

    k_records = periodic(krec)
    v_records = periodic(vrec)
    mean_q = torch.from_numpy(np.ascontiguousarray(mq[0, :, 0])).to(DEV)[None, :, None, :]
    mean_q = mean_q.expand(B, HKV, T_CAP // W, D).contiguous()
    mean_s = torch.from_numpy(np.ascontiguousarray(ms[0, :, 0].view(np.int16))).to(DEV)[None, :, None]
    mean_s = mean_s.expand(B, HKV, T_CAP // W).contiguous()
    assert k_records.numel() * k_records.element_size() > 2 ** 31

    lens = [T_CAP, T_CAP - W * 4099, T_CAP // 2, W]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out = torch.empty((B, HKV * G, D), dtype=torch.float32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, HKV * G, HKV, T_CAP), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dq.dq_decode_attention(gt, gt, q.to(DEV), k_records, mean_q, mean_s, v_records, seq, out, ws, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    del k_records, v_records, mean_q, mean_s
    torch.cuda.empty_cache()

    # the oracle over one period
    k_unit = np.broadcast_to(krec, (B, HKV, W, C)).copy()
    v_unit = np.broadcast_to(vrec, (B, HKV, W, C)).copy()
    ksym, ks, ko, okk = kv.decode_records(k_unit, ot, D)
    vsym, vs, vo, okv = kv.decode_records(v_unit, ot, D)
    assert okk.all() and okv.all()
    mean = kmean.dequantize_mean(np.broadcast_to(mq, (B, HKV, 1, D)).copy(),
                                 np.broadcast_to(ms, (B, HKV, 1)).copy())
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q)), ksym, ks, ko, mean,
                                     vsym, vs, vo, [W] * B, G, 1 / np.sqrt(D))
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got - ref) / scale)) < TOL
