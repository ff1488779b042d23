"""rANS coder and the fixed-size record (oracle).

TEST INFRASTRUCTURE ONLY -- see the package header.

What the paper fixes
--------------------
* Eq. (rans): Enc(x, m) = floor(x / f_m) 2**p + (x mod f_m) + c_m and
  Dec(x, m) = f_m floor(x / 2**p) + (x mod 2**p) - c_m; z = x mod 2**p picks the
  symbol whose interval [c_m, c_m + f_m) holds z; streams are encoded backwards
  so decoding runs in the original order (Sec. 3.1).
* Alg. 2: the state is the little-endian integer in the first sigma/8 bytes of
  the container; after each symbol, while x < L, x = (x << 8) | next byte.
* Eq. (budget), App. A: every stream occupies exactly C bytes, so its address
  follows from the token index.

Readings
--------
* R1 L = 2**21: the state lives in [2**21, 2**29) and is stored as 32 bits
  (sigma = 32).  For p <= 12 a decode step reads at most two bytes.  The
  number of emitted bytes does not depend on L (the stored state always
  carries log2 L bits of the initial value); 2**21 leaves room to keep the
  state scaled by 8 in a 32-bit register.
* R2 the encoder starts from x = L and, before encoding symbol m, emits the low
  byte and shifts while x >= ((L >> p) << 8) f_m, which keeps x in [L, 256 L).
* R3 record layout (C bytes): fp16 scale (LE), fp16 offset (LE), final state
  (LE 32), the emitted bytes in the order the decoder reads them, zero padding.
"""

from __future__ import annotations

import numpy as np

from .tables import Tables, HEADER_BYTES

RANS_L = 1 << 21
STATE_BYTES = 4
PAYLOAD_OFFSET = HEADER_BYTES + STATE_BYTES


def encode(sym: np.ndarray, tab: Tables):
    """Backward rANS encode of streams sym[S, n].

    Returns (state uint64 [S], out uint8 [S, cap], length int [S]) where
    out[s, :length] are the emitted bytes in decode order.
    """
    S, n = sym.shape
    p = tab.p
    x = np.full(S, RANS_L, dtype=np.uint64)
    cap = 2 * n + 8
    emitted = np.zeros((S, cap), dtype=np.uint8)
    count = np.zeros(S, dtype=np.int64)
    rows = np.arange(S)
    xmax_unit = np.uint64((RANS_L >> p) << 8)
    for j in range(n - 1, -1, -1):
        m = sym[:, j]
        f = tab.freq[m].astype(np.uint64)
        c = tab.cum[m].astype(np.uint64)
        xmax = xmax_unit * f
        while True:
            need = x >= xmax
            if not need.any():
                break
            idx = rows[need]
            emitted[idx, count[idx]] = (x[idx] & np.uint64(0xFF)).astype(np.uint8)
            count[idx] += 1
            x[idx] = x[idx] >> np.uint64(8)
        x = (x // f) * np.uint64(1 << p) + (x % f) + c
    out = np.zeros_like(emitted)
    for s in range(S):
        k = int(count[s])
        if k:
            out[s, :k] = emitted[s, :k][::-1]
    return x, out, count


def decode(records: np.ndarray, tab: Tables, n: int):
    """Alg. 2 on records[S, C]: returns (sym [S, n], final x [S], ptr [S]).

    Renormalization reads stop at the end of the C-byte record, so a
    malformed record terminates and shows up as a final state different from L
    (a well-formed record never reaches its end before the last symbol).
    """
    S, C = records.shape
    p = tab.p
    mask = np.uint64((1 << p) - 1)
    rec = records.astype(np.uint64)
    x = (rec[:, 4] | (rec[:, 5] << np.uint64(8)) | (rec[:, 6] << np.uint64(16))
         | (rec[:, 7] << np.uint64(24)))
    ptr = np.full(S, PAYLOAD_OFFSET, dtype=np.int64)
    rows = np.arange(S)
    sym = np.zeros((S, n), dtype=np.int64)
    for j in range(n):
        z = (x & mask).astype(np.int64)
        m = tab.sym_of_z[z]
        sym[:, j] = m
        f = tab.freq[m].astype(np.uint64)
        c = tab.cum[m].astype(np.uint64)
        x = f * (x >> np.uint64(p)) + z.astype(np.uint64) - c
        while True:
            need = (x < np.uint64(RANS_L)) & (ptr < C)
            if not need.any():
                break
            idx = rows[need]
            x[idx] = (x[idx] << np.uint64(8)) | rec[idx, ptr[idx]]
            ptr[idx] += 1
    return sym, x, ptr


def fp16_bits(v: np.ndarray) -> np.ndarray:
    return np.asarray(v, dtype=np.float16).view(np.uint16)


def pack(s16: np.ndarray, o16: np.ndarray, state: np.ndarray, body: np.ndarray,
         length: np.ndarray, C: int) -> np.ndarray:
    """Reading R3: [s16][o16][state LE32][body[:length]][zeros] -> uint8 [S, C]."""
    S = state.shape[0]
    rec = np.zeros((S, C), dtype=np.uint8)
    sb = fp16_bits(s16).astype(np.uint32)
    ob = fp16_bits(o16).astype(np.uint32)
    st = state.astype(np.uint64)
    rec[:, 0] = sb & 0xFF
    rec[:, 1] = sb >> 8
    rec[:, 2] = ob & 0xFF
    rec[:, 3] = ob >> 8
    for k in range(4):
        rec[:, 4 + k] = ((st >> np.uint64(8 * k)) & np.uint64(0xFF)).astype(np.uint8)
    for s in range(S):
        k = int(length[s])
        rec[s, PAYLOAD_OFFSET:PAYLOAD_OFFSET + k] = body[s, :k]
    return rec


def unpack_header(records: np.ndarray):
    """(s16, o16) as float16 arrays from records[S, C]."""
    r = records.astype(np.uint16)
    s = (r[:, 0] | (r[:, 1] << 8)).astype(np.uint16).view(np.float16)
    o = (r[:, 2] | (r[:, 3] << 8)).astype(np.uint16).view(np.float16)
    return s, o
