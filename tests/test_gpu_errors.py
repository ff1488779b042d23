"""Argument checks of the C ABI: every unsupported or inconsistent call is
rejected with its error code before anything is launched.

The calls go straight to libdq's C functions (the Python binding would stop
most of them earlier).  Every buffer passed is large enough for any launch the
arguments could describe, so that even a missing check could not make a kernel
read or write out of bounds.
"""

import ctypes

import pytest
import torch

pytestmark = pytest.mark.gpu

BIG = 1 << 24     # bytes per scratch buffer


@pytest.fixture(scope="module")
def dq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_19880_amd as mod
    return mod


@pytest.fixture(scope="module")
def bufs():
    return [torch.zeros(BIG, dtype=torch.uint8, device="cuda") for _ in range(8)]


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _partial(dq, tk, tv, bufs, B=1, Hq=4, Hkv=1, t_cap=256, ws_bytes=None):
    lib = dq._lib._lib
    if ws_bytes is None:
        ws_bytes = BIG
    return lib.dq_decode_attention_partial(
        tk.handle, tv.handle, _p(bufs[0]), B, Hq, Hkv, _p(bufs[1]),
        _p(bufs[2]), _p(bufs[3]), _p(bufs[4]), _p(bufs[5]), t_cap, ctypes.c_float(0.088),
        _p(bufs[6]), ws_bytes, _p(bufs[7]), None)


def test_attention_rejects_unsupported_records(dq, bufs):
    good = dq.Tables(128, 6, 12, 36, 1.4)
    for C in (37, 72):          # not a whole number of dwords; longer than 64 bytes
        t = dq.Tables(128, 6, 12, C, 1.4)
        assert _partial(dq, t, good, bufs) == dq.DQ_ERR_INVALID_ARG
        assert _partial(dq, good, t, bufs) == dq.DQ_ERR_INVALID_ARG
    assert _partial(dq, good, good, bufs) == dq.DQ_OK
    torch.cuda.synchronize()


def test_attention_rejects_other_head_dims(dq, bufs):
    good = dq.Tables(128, 6, 12, 36, 1.4)
    t64 = dq.Tables(64, 6, 12, 24, 1.4)
    assert _partial(dq, t64, good, bufs) == dq.DQ_ERR_INVALID_ARG
    assert _partial(dq, good, t64, bufs) == dq.DQ_ERR_INVALID_ARG


def test_attention_rejects_bad_shapes(dq, bufs):
    t = dq.Tables(128, 6, 12, 36, 1.4)
    assert _partial(dq, t, t, bufs, Hq=6, Hkv=4) == dq.DQ_ERR_INVALID_ARG      # Hq not a multiple of Hkv
    assert _partial(dq, t, t, bufs, Hq=16, Hkv=1) == dq.DQ_ERR_INVALID_ARG     # more than 8 heads per KV head
    assert _partial(dq, t, t, bufs, t_cap=200) == dq.DQ_ERR_INVALID_ARG        # not whole mean windows
    assert _partial(dq, t, t, bufs, t_cap=0) == dq.DQ_ERR_INVALID_ARG
    assert _partial(dq, t, t, bufs, B=0) == dq.DQ_ERR_INVALID_ARG


def test_attention_rejects_short_workspace(dq, bufs):
    t = dq.Tables(128, 6, 12, 36, 1.4)
    need = dq.dq_decode_workspace_bytes(1, 4, 1, 256)
    assert _partial(dq, t, t, bufs, ws_bytes=need - 1) == dq.DQ_ERR_WORKSPACE
    lib = dq._lib._lib
    rc = lib.dq_decode_attention_merge(1, 4, 1, _p(bufs[5]), 256, _p(bufs[6]), need - 1, _p(bufs[0]), None)
    assert rc == dq.DQ_ERR_WORKSPACE
    rc = lib.dq_decode_attention_merge(1, 4, 1, None, 256, _p(bufs[6]), need, _p(bufs[0]), None)
    assert rc == dq.DQ_ERR_INVALID_ARG


def test_residual_calls_reject_bad_arguments(dq, bufs):
    """The window calls (two-call and one-launch forms): misaligned q or ring,
    ring capacity above 256, short workspace, missing output."""
    lib = dq._lib._lib
    need = dq.dq_decode_workspace_bytes(1, 4, 1, 256)

    def res(q_off=0, rk_off=0, r_cap=128, ws_bytes=need):
        return lib.dq_decode_attention_residual(
            ctypes.c_void_p(bufs[0].data_ptr() + q_off), 1, 4, 1, ctypes.c_void_p(bufs[1].data_ptr() + rk_off),
            _p(bufs[2]), _p(bufs[5]), _p(bufs[4]), r_cap, 256, ctypes.c_float(0.088), _p(bufs[6]), ws_bytes, None)

    def fused(q_off=0, rk_off=0, r_cap=128, ws_bytes=need, out=True):
        return lib.dq_decode_attention_merge_residual(
            ctypes.c_void_p(bufs[0].data_ptr() + q_off), 1, 4, 1, ctypes.c_void_p(bufs[1].data_ptr() + rk_off),
            _p(bufs[2]), _p(bufs[5]), _p(bufs[4]), r_cap, 256, ctypes.c_float(0.088), _p(bufs[6]), ws_bytes,
            _p(bufs[3]) if out else None, None)

    for call in (res, fused):
        assert call(q_off=2) == dq.DQ_ERR_INVALID_ARG
        assert call(rk_off=8) == dq.DQ_ERR_INVALID_ARG
        assert call(r_cap=257) == dq.DQ_ERR_INVALID_ARG
        assert call(r_cap=0) == dq.DQ_ERR_INVALID_ARG
        assert call(ws_bytes=need - 1) == dq.DQ_ERR_WORKSPACE
    assert fused(out=False) == dq.DQ_ERR_INVALID_ARG
    torch.cuda.synchronize()


def test_merge_reads_inside_a_workspace_no_partial_wrote(dq):
    """A workspace whose header no partial call wrote (every byte 0x7F: a
    chunk count and size of 0x7F7F7F7F): the merge, the window and the
    one-launch window + merge bound the chunk count by the workspace's own
    capacity, so they read inside it and return."""
    lib = dq._lib._lib
    B, Hq, Hkv, t_cap, r_cap = 2, 8, 2, 512, 128
    need = dq.dq_decode_workspace_bytes(B, Hq, Hkv, t_cap)
    ws = torch.full((need,), 0x7F, dtype=torch.uint8, device="cuda")
    seq = torch.tensor([500, 37], dtype=torch.int32, device="cuda")
    rl = torch.tensor([100, 3], dtype=torch.int32, device="cuda")
    q = torch.zeros((B, Hq, 128), dtype=torch.bfloat16, device="cuda")
    rk = torch.zeros((B, Hkv, r_cap, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((B, Hq, 128), dtype=torch.float32, device="cuda")
    assert lib.dq_decode_attention_merge(B, Hq, Hkv, _p(seq), t_cap, _p(ws), need, _p(out), None) == dq.DQ_OK
    torch.cuda.synchronize()
    assert lib.dq_decode_attention_merge_residual(_p(q), B, Hq, Hkv, _p(rk), _p(rk), _p(seq), _p(rl), r_cap, t_cap,
                                                  ctypes.c_float(0.088), _p(ws), need, _p(out), None) == dq.DQ_OK
    torch.cuda.synchronize()
    assert lib.dq_decode_attention_residual(_p(q), B, Hq, Hkv, _p(rk), _p(rk), _p(seq), _p(rl), r_cap, t_cap,
                                            ctypes.c_float(0.088), _p(ws), need, None) == dq.DQ_OK
    assert lib.dq_decode_attention_merge(B, Hq, Hkv, _p(seq), t_cap, _p(ws), need, _p(out), None) == dq.DQ_OK
    torch.cuda.synchronize()


def test_encode_rejects_bad_ranges(dq, bufs):
    t = dq.Tables(128, 6, 12, 36, 1.4)
    lib = dq._lib._lib

    def enc(t0, n_new, t_cap, keys=True, H=1, B=1):
        mq, ms = (_p(bufs[2]), _p(bufs[3])) if keys else (None, None)
        return lib.dq_encode_kv(t.handle, _p(bufs[0]), 0, 128, 128, B, H, t0, n_new, t_cap,
                                _p(bufs[1]), mq, ms, _p(bufs[7]), None)

    assert enc(0, 256, 128) == dq.DQ_ERR_INVALID_ARG          # past the capacity
    assert enc(64, 128, 256) == dq.DQ_ERR_INVALID_ARG         # keys: windows must be whole
    assert enc(0, 100, 256) == dq.DQ_ERR_INVALID_ARG
    assert enc(0, 128, 200) == dq.DQ_ERR_INVALID_ARG
    assert enc(-128, 128, 256) == dq.DQ_ERR_INVALID_ARG
    assert enc(0, 128, 256, H=0) == dq.DQ_ERR_INVALID_ARG
    assert enc(0, 0, 256) == dq.DQ_OK                         # nothing to do
    mq_only = lib.dq_encode_kv(t.handle, _p(bufs[0]), 0, 128, 128, 1, 1, 0, 128, 256,
                               _p(bufs[1]), _p(bufs[2]), None, _p(bufs[7]), None)
    assert mq_only == dq.DQ_ERR_INVALID_ARG                   # means need both buffers
    torch.cuda.synchronize()


def test_tables_reject_bad_configs(dq):
    with pytest.raises(dq.DqError):
        dq.Tables(128, 16, 12, 36, 1.4)      # infeasible at alpha 1.4 (Tab. 2 marks it "--")
    with pytest.raises(dq.DqError):
        dq.Tables(96, 6, 12, 36, 1.4)        # head_dim not a power of two
    with pytest.raises(dq.DqError):
        dq.Tables(128, 6, 13, 36, 1.4)       # precision above 12 bits
