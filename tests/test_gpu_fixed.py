"""Fixed-width comparator at matched storage (App. B) on the GPU against the
oracle (oracle/fixed.py), through the C ABI.

Bars as in test_gpu_parity.py: records and key means bit-exact; attention
within 2e-3 (row-normalized) of the oracle's fp64 folded attention over the
oracle's own fixed-width records.
"""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, fixed, kmean, kv

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


def _inputs(B, T, H, G, d, seed):
    wl = wlmod.workload("b1_t4k")
    w2 = wlmod.Workload("fixed", B, T, H * G, H, 4, wl.k, wl.v, head_dim=d)
    return wlmod.make_k(w2, seed), wlmod.make_v(w2, seed), wlmod.make_q(w2, seed)


@pytest.mark.parametrize("d,C", [(128, 36), (128, 32), (128, 48), (64, 28), (256, 72)])
def test_fixed_encode_bit_exact(dq, d, C):
    B, T, H = 2, 256, 2
    k, v, _ = _inputs(B, T, H, 1, d, 51)
    kb, vb = wlmod.bf16_bits(k), wlmod.bf16_bits(v)
    krec, mq, ms, _ = fixed.encode_keys(kb, C)
    vrec, _ = fixed.encode_values(vb, C)
    grk = torch.full((B, H, T, C), 0xAB, dtype=torch.uint8, device=DEV)
    grv = torch.full((B, H, T, C), 0xAB, dtype=torch.uint8, device=DEV)
    gmq = torch.zeros((B, H, T // 128, d), dtype=torch.int8, device=DEV)
    gms = torch.zeros((B, H, T // 128), dtype=torch.int16, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    dq.dq_encode_kv_fixed(d, C, kd[:, :128], 0, T, grk, gmq, gms, status)
    dq.dq_encode_kv_fixed(d, C, kd[:, 128:], 128, T, grk, gmq, gms, status)
    dq.dq_encode_kv_fixed(d, C, vd[:, :77], 0, T, grv, None, None, status)
    dq.dq_encode_kv_fixed(d, C, vd[:, 77:], 77, T, grv, None, None, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert np.array_equal(grk.cpu().numpy(), krec)
    assert np.array_equal(grv.cpu().numpy(), vrec)
    assert np.array_equal(gmq.cpu().numpy(), mq)
    assert np.array_equal(gms.cpu().numpy().view(np.uint16), ms.view(np.uint16))


@pytest.mark.parametrize("G", [4, 2, 1])
def test_fixed_attention_matches_oracle(dq, G):
    B, T, H, d, C = 4, 512, 2, 128, 36
    k, v, q = _inputs(B, T, H, G, d, 52 + G)
    krec, mq, ms, _ = fixed.encode_keys(wlmod.bf16_bits(k), C)
    vrec, _ = fixed.encode_values(wlmod.bf16_bits(v), C)
    lens = [T, 0, 65, 300]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, H * G, H, T), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, H * G, 128), dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    grk, grv = torch.from_numpy(krec).to(DEV), torch.from_numpy(vrec).to(DEV)
    gmq, gms = torch.from_numpy(mq).to(DEV), torch.from_numpy(ms.view(np.int16)).to(DEV)
    outs = []
    for _ in range(2):
        dq.dq_decode_attention_fixed_partial(q.to(DEV), grk, gmq, gms, grv, seq, ws, status=status)
        dq.dq_decode_attention_merge(B, H * G, H, seq, T, ws, out)
        torch.cuda.synchronize()
        outs.append(out.cpu().clone())
    assert int(status.item()) == 0
    assert torch.equal(outs[0], outs[1])
    ksym, ks, ko = fixed.unpack(krec, d, 2)
    vsym, vs, vo = fixed.unpack(vrec, d, 2)
    ref = attention.attention_folded(kv.bf16_to_f64(wlmod.bf16_bits(q)), ksym, ks, ko,
                                     kmean.dequantize_mean(mq, ms), vsym, vs, vo, lens, G, 1 / np.sqrt(d))
    got = outs[0].numpy().astype(np.float64)
    assert np.all(got[1] == 0.0)
    assert _rel_err(got[[0, 2, 3]], ref[[0, 2, 3]]) < TOL


def test_fixed_entry_points_reject_bad_arguments(dq):
    lib = dq._lib._lib
    big = torch.zeros(1 << 22, dtype=torch.uint8, device=DEV)
    p = big.data_ptr()
    assert dq.dq_fixed_bits(128, 4) == 0 and dq.dq_fixed_bits(128, 40) == 2
    assert lib.dq_encode_kv_fixed(96, 36, p, 0, 96, 96, 1, 1, 0, 128, 256, p, None, None, p, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_encode_kv_fixed(128, 4, p, 0, 128, 128, 1, 1, 0, 128, 256, p, None, None, p, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_encode_kv_fixed(128, 36, p, 0, 128, 128, 1, 1, 0, 100, 256, p, p, p, p, None) == dq.DQ_ERR_INVALID_ARG

    def attn(Hq=4, Hkv=1, t_cap=256, ws_bytes=1 << 22):
        return lib.dq_decode_attention_fixed_partial(p, 1, Hq, Hkv, p, p, p, p, p, t_cap, 0.088, p, ws_bytes, p,
                                                     None)

    assert attn(Hq=8) == dq.DQ_ERR_INVALID_ARG
    assert attn(t_cap=200) == dq.DQ_ERR_INVALID_ARG
    assert attn(ws_bytes=16) == dq.DQ_ERR_WORKSPACE
