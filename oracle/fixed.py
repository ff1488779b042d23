"""Fixed-width comparator at matched storage (App. B) (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

What the paper fixes
--------------------
* App. B sets D-Quant's entropy-coded record against a fixed-width code
  given the same bytes.  Everything before the coder is shared (rotation, the
  keys' 8-bit window means, the per-token min-max grid, the least-squares
  refit, fp16 scale and offset); the fixed-width side rounds every value to its
  nearest level and is charged log2 M bits per symbol.
* Sec. 3 (Background): b bits give exactly 2**b levels; 2-bit codes for 128
  values plus one fp16 scale and one fp16 offset come to 2.25 bits per value.

Readings
--------
* F1 record: the same C bytes as a D-Quant record, [fp16 s][fp16 o] then the
  symbols at b = floor(8 (C - 4) / n) bits each, M = 2**b levels (no rANS
  state: every bit after the header carries symbols).  Symbol j occupies
  payload bits [b j, b j + b), least significant bit first, bit k of the
  payload being bit k mod 8 of byte 4 + k // 8; the rest is zero.  At the
  measured 36-byte, 128-value records b = 2: the paper's INT2 example.
* F3 App. B's own charge: each fixed-width symbol costs the ideal log2 M bits,
  so the comparator takes the largest M with M**n <= 2**(8 (C - 4)) (the
  record less its fp16 scale and offset).  At the per-token operating point
  (n = 1024, 335 / 235-byte records) that is 6 key and 3 value levels, the
  counts App. B states; at 128-value, 36-byte records it is 4, the same as F1.
  Such symbols are an accounting device (6**1024 fills 331 bytes to the
  bit), used for reconstruction error only; F1 is the stored format.
* F2 quantizer: Alg. 1 with each Drift replaced by nearest-level rounding,
  i.e. FitMinMax -> nearest -> Refit -> fp16 -> nearest; "nearest" is
  argmin_m D_im of reading Q1 with ties to the smallest m (Drift's assignment
  at lambda = 0).
"""

from __future__ import annotations

import numpy as np

from . import kv, quantize, rans


def bits_per_symbol(n: int, record_bytes: int) -> int:
    """Reading F1: b = floor(8 (C - 4) / n)."""
    return (8 * (record_bytes - 4)) // n


def ideal_levels(n: int, record_bytes: int) -> int:
    """Reading F3: the largest M with M**n <= 2**(8 (C - 4)) (exact integers)."""
    budget = 1 << (8 * (record_bytes - 4))
    M = 1
    while (M + 1) ** n <= budget:
        M += 1
    return M


def nearest(x: np.ndarray, s: np.ndarray, o: np.ndarray, M: int) -> np.ndarray:
    """argmin_m (x - (o + s m))**2 per value, ties to the smallest m."""
    return np.argmin(quantize.distortion(x, s, o, M), axis=-1).astype(np.int64)


def quantize_streams(x: np.ndarray, M: int):
    """Reading F2 for streams x[S, n] (fp64): (sym [S, n], s16, o16)."""
    s0, o0 = quantize.fit_minmax(x, M)
    m1 = nearest(x, s0, o0, M)
    s1, o1 = quantize.refit(x, m1, s0, o0)
    s16, o16 = quantize.to_fp16(s1), quantize.to_fp16(o1)
    m = nearest(x, s16.astype(np.float64), o16.astype(np.float64), M)
    return m, s16, o16


def pack(sym: np.ndarray, s16: np.ndarray, o16: np.ndarray, b: int, C: int) -> np.ndarray:
    """Reading F1: records uint8 [S, C]."""
    S, n = sym.shape
    rec = np.zeros((S, C), dtype=np.uint8)
    sb = rans.fp16_bits(s16).astype(np.uint32)
    ob = rans.fp16_bits(o16).astype(np.uint32)
    rec[:, 0] = sb & 0xFF
    rec[:, 1] = sb >> 8
    rec[:, 2] = ob & 0xFF
    rec[:, 3] = ob >> 8
    bits = np.zeros((S, 8 * (C - 4)), dtype=np.uint8)
    for i in range(b):
        bits[:, i:n * b:b] = (sym >> i) & 1
    body = np.packbits(bits, axis=1, bitorder="little")
    rec[:, 4:] = body
    return rec


def unpack(records: np.ndarray, n: int, b: int):
    """records [..., C] -> (sym [..., n], s16, o16)."""
    lead = records.shape[:-1]
    flat = records.reshape(-1, records.shape[-1])
    bits = np.unpackbits(flat[:, 4:], axis=1, bitorder="little").astype(np.int64)
    sym = np.zeros((flat.shape[0], n), dtype=np.int64)
    for i in range(b):
        sym |= bits[:, i:n * b:b] << i
    s16, o16 = rans.unpack_header(flat)
    return sym.reshape(*lead, n), s16.reshape(lead), o16.reshape(lead)


def encode_keys(k_bits: np.ndarray, record_bytes: int, window: int = 128):
    """Keys [B, T, H, d] -> (records [B, H, T, C], mean_q, mean_scale, sym [B, H, T, d]),
    with the same per-head rotation and window means as the D-Quant encoder."""
    B, T, H, d = k_bits.shape
    b = bits_per_symbol(d, record_bytes)
    x, mq, ms = kv._key_streams(k_bits, window)
    sym, s16, o16 = quantize_streams(x.reshape(B * H * T, d), 1 << b)
    rec = pack(sym, s16, o16, b, record_bytes)
    return rec.reshape(B, H, T, record_bytes), mq, ms, sym.reshape(B, H, T, d)


def encode_values(v_bits: np.ndarray, record_bytes: int):
    """Values [B, T, H, d] -> (records [B, H, T, C], sym)."""
    B, T, H, d = v_bits.shape
    b = bits_per_symbol(d, record_bytes)
    x = kv.rotate(v_bits).transpose(0, 2, 1, 3).reshape(B * H * T, d)
    sym, s16, o16 = quantize_streams(x, 1 << b)
    rec = pack(sym, s16, o16, b, record_bytes)
    return rec.reshape(B, H, T, record_bytes), sym.reshape(B, H, T, d)
