"""The BF16 comparator (plain decode attention over an uncompressed cache) on
the GPU against the oracle's attention over raw tokens (a residual window of
full length, reading A3), within 2e-3 row-normalized."""

import numpy as np
import pytest
import torch

import dq_workloads as wlmod
from oracle import attention, kv

pytestmark = pytest.mark.gpu

TOL = 2e-3
DEV = "cuda"


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


@pytest.mark.parametrize("G", [1, 4, 8])
def test_bf16_decode_matches_oracle(dq, G):
    wl = wlmod.workload("b1_t4k")
    B, Hkv, t_cap = 3, 2, 1024
    lens = [1000, 0, 577]
    w2 = wlmod.Workload("bf16", B, t_cap, Hkv * G, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, 31)                       # [B, T, H, d]
    v = wlmod.make_v(w2, 31)
    q = wlmod.make_q(w2, 31)
    kd = k.permute(0, 2, 1, 3).contiguous().to(DEV)  # [B, H, T, d]
    vd = v.permute(0, 2, 1, 3).contiguous().to(DEV)
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hkv * G, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hkv * G, 128), dtype=torch.float32, device=DEV)
    dq.dq_bf16_decode_attention_partial(q.to(DEV), kd, vd, seq, ws)
    dq.dq_decode_attention_merge(B, Hkv * G, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    rk = np.moveaxis(kv.bf16_to_f64(wlmod.bf16_bits(k)), 1, 2)
    rv = np.moveaxis(kv.bf16_to_f64(wlmod.bf16_bits(v)), 1, 2)
    empty = np.zeros((B, Hkv, 0, 128))
    ref = attention.attention_with_residual(kv.bf16_to_f64(wlmod.bf16_bits(q)), empty, empty, [0] * B,
                                            rk, rv, lens, G, 1 / np.sqrt(128))
    assert np.all(got[1] == 0.0)
    scale = np.max(np.abs(ref[[0, 2]]), axis=-1, keepdims=True)
    assert float(np.max(np.abs(got[[0, 2]] - ref[[0, 2]]) / scale)) < TOL
