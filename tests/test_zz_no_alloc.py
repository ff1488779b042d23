"""dq_decode_attention_no_alloc, the decode step whose split-K workspace is
the library's static per-device scratch array, against dq_decode_attention
with a caller workspace: the same kernels and chunk plan, so the outputs must
be equal bit for bit.  Two calls in a row, the second on a smaller input
(fewer sequences, shorter context, another GQA group and coding), then the
first again; ragged and empty sequences; the size limit of the array on both
sides (rejected with DQ_ERR_WORKSPACE, launching nothing, just above it)."""

import pytest
import torch

import bench
import dq_workloads as wlmod
import paper_2609_19880_amd as dq

pytestmark = pytest.mark.gpu

SEED = 5


def _cache(name, context, batch):
    wl = wlmod.workload(name).with_context(context, batch=batch)
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, torch.device("cuda"))
    return wl, tk, tv, cache


def _both(wl, tk, tv, cache, lens, qseed):
    dev = torch.device("cuda")
    q = wlmod.make_q(wl, qseed, device=dev)
    seq = torch.tensor(lens, dtype=torch.int32, device=dev)
    got = torch.full((wl.batch, wl.q_heads, wl.head_dim), float("nan"), device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    dq.dq_decode_attention_no_alloc(tk, tv, q, cache.k_records, cache.k_mean_q, cache.k_mean_scale,
                                    cache.v_records, seq, got, status=status)
    torch.cuda.synchronize()
    ref = cache.attend(q, seq)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert int(cache.status.item()) == 0
    return got, ref


@pytest.fixture(scope="module")
def caches():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return {"big": _cache("b1_t4k", 4096, 4), "small": _cache("b32_t32k_g8", 1024, 2)}


def test_no_alloc_equals_workspace_path_twice(caches):
    # first call: 4 sequences x 4096 tokens, G = 4, shared 36-byte coding
    got, ref = _both(*caches["big"], [4096, 1000, 0, 2113], 11)
    assert torch.equal(got, ref)
    assert torch.all(got[2] == 0)
    # second call, smaller: 2 sequences x 1024 tokens, G = 8, K 48 / V 32 bytes
    got, ref = _both(*caches["small"], [1024, 300], 12)
    assert torch.equal(got, ref)
    assert torch.isfinite(got).all()
    # the first input again, with another query: nothing of the last call leaks
    got, ref = _both(*caches["big"], [17, 4096, 129, 0], 13)
    assert torch.equal(got, ref)


def test_no_alloc_size_limit():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # t_cap 128: one chunk and four residual slots, so the workspace is
    # 256 + 520 B Hq 5 bytes; 64 query heads: B = 50 fits in 8 MiB, B = 51 does not
    wl, tk, tv, cache = _cache("b32_t32k_g8", 128, 51)
    dev = torch.device("cuda")
    q = wlmod.make_q(wl, 21, device=dev)
    seq = torch.full((51,), 128, dtype=torch.int32, device=dev)
    out = torch.zeros((51, 64, 128), dtype=torch.float32, device=dev)
    with pytest.raises(dq.DqError) as ei:
        dq.dq_decode_attention_no_alloc(tk, tv, q, cache.k_records, cache.k_mean_q, cache.k_mean_scale,
                                        cache.v_records, seq, out)
    assert ei.value.code == dq.DQ_ERR_WORKSPACE
    assert "scratch" in dq.dq_last_error()
    torch.cuda.synchronize()
    assert torch.all(out == 0)          # nothing was launched

    n = 50
    assert 256 + 520 * n * 64 * 5 <= dq.DQ_NO_ALLOC_SCRATCH_BYTES < 256 + 520 * (n + 1) * 64 * 5
    sub = (cache.k_records[:n].contiguous(), cache.k_mean_q[:n].contiguous(),
           cache.k_mean_scale[:n].contiguous(), cache.v_records[:n].contiguous())
    got = torch.empty((n, 64, 128), dtype=torch.float32, device=dev)
    dq.dq_decode_attention_no_alloc(tk, tv, q[:n].contiguous(), *sub[:3], sub[3], seq[:n], got)
    ref = torch.empty_like(got)
    ws = torch.empty(dq.dq_decode_workspace_bytes(n, 64, 8, 128), dtype=torch.uint8, device=dev)
    dq.dq_decode_attention(tk, tv, q[:n].contiguous(), *sub[:3], sub[3], seq[:n], ref, ws)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
