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


def _bf16_step(dq, q, kd, vd, lens, Hq, Hkv, t_cap):
    B = q.shape[0]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws = torch.empty(dq.dq_decode_workspace_bytes(B, Hq, Hkv, t_cap), dtype=torch.uint8, device=DEV)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=DEV)
    dq.dq_bf16_decode_attention_partial(q, kd, vd, seq, ws)
    dq.dq_decode_attention_merge(B, Hq, Hkv, seq, t_cap, ws, out)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _oracle_head(q, k, v, b, h, G, T):
    """Oracle attention of the G query heads of KV head h of sequence b (k, v [B, H, T, d] bf16 on the host)."""
    qf = kv.bf16_to_f64(wlmod.bf16_bits(q[b:b + 1, h * G:(h + 1) * G]))
    rk = kv.bf16_to_f64(wlmod.bf16_bits(k[b:b + 1, h:h + 1, :T]))
    rv = kv.bf16_to_f64(wlmod.bf16_bits(v[b:b + 1, h:h + 1, :T]))
    empty = np.zeros((1, 1, 0, 128))
    return attention.attention_with_residual(qf, empty, empty, [0], rk, rv, [T], G, 1 / np.sqrt(128))[0]


@pytest.mark.parametrize("G", [4, 8])
def test_bf16_rows_past_length_are_ignored(dq, G):
    """Rows past a sequence's length may hold anything (here NaN and inf
    patterns): the output is bit-identical to the one with those rows zeroed,
    and matches the oracle."""
    wl = wlmod.workload("b1_t4k")
    B, Hkv, t_cap = 2, 2, 1024
    lens = [999, 130]
    w2 = wlmod.Workload("bf16", B, t_cap, Hkv * G, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, 41).permute(0, 2, 1, 3).contiguous()     # [B, H, T, d]
    v = wlmod.make_v(w2, 41).permute(0, 2, 1, 3).contiguous()
    q = wlmod.make_q(w2, 41)
    kz, vz, kn, vn = k.clone(), v.clone(), k.clone(), v.clone()
    nan = torch.tensor([0x7FC0], dtype=torch.int16).view(torch.bfloat16)
    inf = torch.tensor([0x7F80], dtype=torch.int16).view(torch.bfloat16)
    for b, T in enumerate(lens):
        kz[b, :, T:] = 0
        vz[b, :, T:] = 0
        kn[b, :, T:] = nan
        vn[b, :, T::2] = inf
        vn[b, :, T + 1::2] = nan
    got_z = _bf16_step(dq, q.to(DEV), kz.to(DEV), vz.to(DEV), lens, Hkv * G, Hkv, t_cap)
    got_n = _bf16_step(dq, q.to(DEV), kn.to(DEV), vn.to(DEV), lens, Hkv * G, Hkv, t_cap)
    assert np.array_equal(got_z, got_n)
    for b, T in enumerate(lens):
        for h in range(Hkv):
            ref = _oracle_head(q, k, v, b, h, G, T)
            got = got_n[b, h * G:(h + 1) * G]
            scale = np.max(np.abs(ref), axis=-1, keepdims=True)
            assert float(np.max(np.abs(got - ref) / scale)) < TOL


def test_bf16_full_context_sampled(dq):
    """The headline shape's per-sequence context (32768 tokens, 32 / 8 heads)
    in the launch configuration the comparator is timed in: two sequences,
    one ragged, every KV head checked against the oracle."""
    B, Hq, Hkv, t_cap = 2, 32, 8, 32768
    lens = [32768, 20001]
    wl = wlmod.workload("b16_t32k")
    w2 = wlmod.Workload("bf16", B, t_cap, Hq, Hkv, 4, wl.k, wl.v)
    k = wlmod.make_k(w2, 43).permute(0, 2, 1, 3).contiguous()
    v = wlmod.make_v(w2, 43).permute(0, 2, 1, 3).contiguous()
    q = wlmod.make_q(w2, 43)
    got = _bf16_step(dq, q.to(DEV), k.to(DEV), v.to(DEV), lens, Hq, Hkv, t_cap)
    G = Hq // Hkv
    for b, T in enumerate(lens):
        for h in range(Hkv):
            ref = _oracle_head(q, k, v, b, h, G, T)
            scale = np.max(np.abs(ref), axis=-1, keepdims=True)
            assert float(np.max(np.abs(got[b, h * G:(h + 1) * G] - ref) / scale)) < TOL
