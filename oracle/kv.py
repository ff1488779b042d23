"""The append path over a KV tensor, and its inverse (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

Pipeline of Fig. 1 / Sec. 4.2, one stream per (token, KV head):
  bf16 -> fp64 -> Hadamard (hadamard.fwht) -> keys: minus the dequantized
  window mean (kmean) -> Alg. 1 (quantize) -> rANS record (rans).

Reading K2 (streams over all KV heads, the paper's default grouping):
Sec. 4.1 defines a stream as the values of one token's key or value tensor,
and Sec. 4.5 / Sec. 5.1 make that one group of H_kv d = 1024 values spanning
every KV head.  The stream takes the heads in order, each in its rotated
channel order (value j = h d + c), which is the order the decoder consumes
them one KV head at a time.  Rotation and the key window mean stay per head;
the affine (s, o) and the record are per token.  The *_tokenwise functions
build these streams; with H_kv = 1 they are the per-head streams.

Reading V0 (prerotated tensors, Sec. 4.2: the value rotation can be folded
into the projection weights offline): with rotate=False the input already is
the rotated vector and is coded as it is, with no Hadamard.

Reading K1 (container overflow): the drift guarantees the ideal cost
sum r <= B; should the rANS bytes still exceed the record (8 + E > C), the
budget is lowered by 8 bits and the second Drift and the coder are run again,
until it fits.  An encode error is raised if the budget would fall below the
cheapest possible stream.
"""

from __future__ import annotations

import numpy as np

from . import hadamard, kmean, quantize, rans
from .tables import Tables, Q16

BATCH = 2048


class EncodeError(RuntimeError):
    pass


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp64, exact."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def encode_streams(x: np.ndarray, tab: Tables):
    """Alg. 1 + rANS for streams x[S, n] (fp64).

    Returns (records uint8 [S, C], sym int64 [S, n], s16, o16, budget int64 [S])
    where budget is the Q16 budget the final assignment was made under.
    """
    if not tab.feasible:
        raise EncodeError("infeasible table: n * min cost exceeds the budget")
    S, n = x.shape
    C = tab.record_bytes
    recs = np.zeros((S, C), dtype=np.uint8)
    syms = np.zeros((S, n), dtype=np.int64)
    s16s = np.zeros(S, dtype=np.float16)
    o16s = np.zeros(S, dtype=np.float16)
    budgets = np.zeros(S, dtype=np.int64)
    floor_budget = n * int(tab.cost.min())
    for a in range(0, S, BATCH):
        xb = x[a:a + BATCH]
        s16, o16 = quantize.first_pass(xb, tab)
        if not (np.all(np.isfinite(s16)) and np.all(np.isfinite(o16))):
            raise EncodeError("scale or offset overflows fp16")
        budget = np.full(xb.shape[0], tab.budget_q16, dtype=np.int64)
        todo = np.arange(xb.shape[0])
        while todo.size:
            m = quantize.final_drift(xb[todo], s16[todo], o16[todo], tab, budget[todo])
            state, body, length = rans.encode(m, tab)
            fits = rans.PAYLOAD_OFFSET + length <= C
            ok = todo[fits]
            rec = rans.pack(s16[ok], o16[ok], state[fits], body[fits], length[fits], C)
            recs[a + ok] = rec
            syms[a + ok] = m[fits]
            budgets[a + ok] = budget[ok]
            todo = todo[~fits]
            budget[todo] -= 8 * Q16
            if todo.size and budget[todo].min() < floor_budget:
                raise EncodeError("record overflow could not be resolved")
        s16s[a:a + BATCH] = s16
        o16s[a:a + BATCH] = o16
    return recs, syms, s16s, o16s, budgets


def rotate(bits: np.ndarray, on: bool = True) -> np.ndarray:
    """bf16 [..., d] -> rotated fp64 [..., d] (on=False: fp64 as given, reading V0)."""
    return hadamard.fwht(bf16_to_f64(bits)) if on else bf16_to_f64(bits)


def encode_keys(k_bits: np.ndarray, tab: Tables, window: int = 128, rotate_on: bool = True):
    """Keys [B, T, H, d] (bf16 bits) -> (records [B, H, T, C],
    mean_q int8 [B, H, T/W, d], mean_scale fp16 [B, H, T/W], sym [B, H, T, d])."""
    B, T, H, d = k_bits.shape
    x, mq, ms = _key_streams(k_bits, window, rotate_on)
    recs, syms, _, _, _ = encode_streams(x.reshape(B * H * T, d), tab)
    C = tab.record_bytes
    return (recs.reshape(B, H, T, C), mq, ms, syms.reshape(B, H, T, d))


def encode_values(v_bits: np.ndarray, tab: Tables, rotate_on: bool = True):
    """Values [B, T, H, d] (bf16 bits) -> (records [B, H, T, C], sym)."""
    B, T, H, d = v_bits.shape
    x = rotate(v_bits, rotate_on).transpose(0, 2, 1, 3).reshape(B * H * T, d)
    recs, syms, _, _, _ = encode_streams(x, tab)
    return recs.reshape(B, H, T, tab.record_bytes), syms.reshape(B, H, T, d)


def decode_records(records: np.ndarray, tab: Tables, n: int):
    """records [..., C] -> (sym [..., n], s16, o16, ok [...]).

    ok is False where the decoder does not end in state L with its pointer
    inside the record (Alg. 2 invariants).
    """
    lead = records.shape[:-1]
    flat = records.reshape(-1, records.shape[-1])
    sym, x, ptr = rans.decode(flat, tab, n)
    s16, o16 = rans.unpack_header(flat)
    ok = (x == rans.RANS_L) & (ptr <= flat.shape[1])
    return (sym.reshape(*lead, n), s16.reshape(lead), o16.reshape(lead), ok.reshape(lead))


def _key_streams(k_bits: np.ndarray, window: int, rotate_on: bool = True):
    """Rotated keys minus their dequantized window means, [B, H, T, d],
    with the INT8 means and their fp16 scales."""
    B, T, H, d = k_bits.shape
    if T % window:
        raise ValueError("token count must be a multiple of the mean window")
    y = rotate(k_bits, rotate_on).transpose(0, 2, 1, 3)          # [B, H, T, d]
    nw = T // window
    yw = y.reshape(B, H, nw, window, d)
    mu = kmean.window_mean(yw)
    mq, ms = kmean.quantize_mean(mu)
    if not np.all(np.isfinite(ms.astype(np.float64))):
        raise EncodeError("key mean scale overflows fp16")
    mu_hat = kmean.dequantize_mean(mq, ms)
    return (yw - mu_hat[:, :, :, None, :]).reshape(B, H, T, d), mq, ms


def encode_keys_tokenwise(k_bits: np.ndarray, tab: Tables, window: int = 128, rotate_on: bool = True):
    """Keys [B, T, H, d] -> one stream of n = H d values per token (reading K2).

    Returns (records [B, T, C], mean_q int8 [B, H, T/W, d],
    mean_scale fp16 [B, H, T/W], sym [B, T, H d]).
    """
    B, T, H, d = k_bits.shape
    if tab.n != H * d:
        raise ValueError("the table's stream length must be H * d")
    x, mq, ms = _key_streams(k_bits, window, rotate_on)
    x = x.transpose(0, 2, 1, 3).reshape(B * T, H * d)
    recs, syms, _, _, _ = encode_streams(x, tab)
    return recs.reshape(B, T, tab.record_bytes), mq, ms, syms.reshape(B, T, H * d)


def encode_values_tokenwise(v_bits: np.ndarray, tab: Tables, rotate_on: bool = True):
    """Values [B, T, H, d] -> (records [B, T, C], sym [B, T, H d]) (reading K2)."""
    B, T, H, d = v_bits.shape
    if tab.n != H * d:
        raise ValueError("the table's stream length must be H * d")
    x = rotate(v_bits, rotate_on).reshape(B * T, H * d)
    recs, syms, _, _, _ = encode_streams(x, tab)
    return recs.reshape(B, T, tab.record_bytes), syms.reshape(B, T, H * d)


def tokenwise_as_heads(sym: np.ndarray, s16: np.ndarray, o16: np.ndarray, H: int):
    """Token streams (sym [B, T, H d], s16 / o16 [B, T]) viewed per KV head:
    (sym [B, H, T, d], s16 [B, H, T], o16 [B, H, T]); every head of a token
    shares the token's (s, o)."""
    B, T, n = sym.shape
    d = n // H
    sh = sym.reshape(B, T, H, d).transpose(0, 2, 1, 3)
    s = np.broadcast_to(s16[:, None, :], (B, H, T))
    o = np.broadcast_to(o16[:, None, :], (B, H, T))
    return sh, s, o
