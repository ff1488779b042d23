"""A decode step captured in a HIP graph (torch.cuda.CUDAGraph around the
library's partial, residual and merge calls) and replayed, as a serving loop
replays its step to drop the per-launch host work.  Every replay, with a new
query copied into the captured buffer and the program's own eager steps and
synchronizations in between, must equal the eager step bit for bit; ragged
and empty sequences included.  Per-(token, KV head) and per-token streams."""

import pytest
import torch

import bench
import dq_workloads as wlmod
import paper_2609_19880_amd as dq

pytestmark = pytest.mark.gpu

SEED = 3
REPLAYS = 4


def _capture(step):
    """Warm up on a side stream, then capture step() into a graph."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def _check_replays(wl, cache, lens, extra=None, zero_rows=(), finish=None):
    dev = torch.device("cuda")
    q, _, out = bench.step_inputs(wl, SEED, dev)
    seq = torch.tensor(lens, dtype=torch.int32, device=dev)
    static_q, static_out = q.clone(), torch.empty_like(out)

    def step(qq, oo):
        cache.partial(qq, seq)
        if extra is not None:
            extra(qq)
        if finish is not None:
            finish(qq, oo)
        else:
            cache.merge(seq, oo)

    g = _capture(lambda: step(static_q, static_out))
    for i in range(REPLAYS):
        qi = wlmod.make_q(wl, SEED + 10 + i, device=dev)
        static_q.copy_(qi)
        g.replay()
        torch.cuda.synchronize()
        got = static_out.clone()
        ref = torch.empty_like(out)
        step(qi, ref)                       # eager step between the replays
        torch.cuda.synchronize()
        assert torch.equal(got, ref), i
        assert torch.isfinite(got).all()
        for b in zero_rows:               # no tokens at all: the output is 0
            assert torch.all(got[b] == 0)
    assert int(cache.status.item()) == 0


@pytest.fixture(scope="module")
def head_cache():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = wlmod.workload("b1_t4k").with_context(4096, batch=4)
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, torch.device("cuda"))
    return wl, cache


def test_graph_replay_per_head_streams(head_cache):
    wl, cache = head_cache
    _check_replays(wl, cache, [4096, 1000, 0, 2113], zero_rows=(2,))


def test_graph_replay_with_residual_window(head_cache):
    wl, cache = head_cache
    dev = torch.device("cuda")
    B, Hkv, d = wl.batch, wl.kv_heads, wl.head_dim
    g = torch.Generator(device=dev)
    g.manual_seed(SEED)
    rk = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
    rv = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
    lens = [4096, 1000, 0, 2113]
    seq = torch.tensor(lens, dtype=torch.int32, device=dev)
    rl = torch.tensor([37, 128, 5, 0], dtype=torch.int32, device=dev)   # sequence 2: raw tokens only
    _check_replays(wl, cache, lens,
                   extra=lambda qq: dq.dq_decode_attention_residual(qq, rk, rv, seq, rl, cache.t_cap,
                                                                    cache.workspace))


def test_graph_replay_merge_with_residual_window(head_cache):
    """The one-launch window + merge in the captured step."""
    wl, cache = head_cache
    dev = torch.device("cuda")
    B, Hkv, d = wl.batch, wl.kv_heads, wl.head_dim
    g = torch.Generator(device=dev)
    g.manual_seed(SEED + 1)
    rk = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
    rv = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
    lens = [4096, 1000, 0, 2113]
    seq = torch.tensor(lens, dtype=torch.int32, device=dev)
    rl = torch.tensor([255, 128, 5, 0], dtype=torch.int32, device=dev)
    _check_replays(wl, cache, lens,
                   finish=lambda qq, oo: dq.dq_decode_attention_merge_residual(qq, rk, rv, seq, rl, cache.t_cap,
                                                                               cache.workspace, oo))


def test_graph_replay_per_token_streams():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = wlmod.workload("b16_t32k_tok").with_context(4096, batch=3)
    tk, tv, cache, _ = bench.fill_cache(wl, SEED, torch.device("cuda"))
    _check_replays(wl, cache, [4096, 0, 1729], zero_rows=(1,))
