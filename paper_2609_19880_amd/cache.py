"""A compressed KV cache for one attention layer: buffers plus the two calls.

torch allocates the device buffers; encoding and attention are the library's
kernels.  Records are stored [batch][kv_heads][t_cap][C] so that the address of
a token's record follows from its index (App. A).
"""

from __future__ import annotations

import torch

from . import _lib


class KVCache:
    def __init__(self, batch: int, kv_heads: int, q_heads: int, t_cap: int, k_tables, v_tables,
                 device="cuda"):
        if t_cap % _lib.DQ_MEAN_WINDOW:
            raise ValueError("t_cap must be a multiple of 128")
        d = k_tables.head_dim
        self.batch, self.kv_heads, self.q_heads, self.t_cap, self.head_dim = batch, kv_heads, q_heads, t_cap, d
        self.k_tables, self.v_tables = k_tables, v_tables
        nw = t_cap // _lib.DQ_MEAN_WINDOW
        self.k_records = torch.zeros((batch, kv_heads, t_cap, k_tables.record_bytes), dtype=torch.uint8, device=device)
        self.v_records = torch.zeros((batch, kv_heads, t_cap, v_tables.record_bytes), dtype=torch.uint8, device=device)
        self.k_mean_q = torch.zeros((batch, kv_heads, nw, d), dtype=torch.int8, device=device)
        self.k_mean_scale = torch.zeros((batch, kv_heads, nw), dtype=torch.int16, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.workspace = torch.empty(
            _lib.dq_decode_workspace_bytes(batch, q_heads, kv_heads, t_cap, d), dtype=torch.uint8, device=device)

    def append(self, k, v, t0: int):
        """Encode bf16 k, v [B, T_new, H, d] as cache tokens [t0, t0 + T_new)."""
        _lib.dq_encode_kv(self.k_tables, k, t0, self.t_cap, self.k_records, self.k_mean_q,
                          self.k_mean_scale, self.status)
        _lib.dq_encode_kv(self.v_tables, v, t0, self.t_cap, self.v_records, None, None, self.status)

    def attend(self, q, seq_lens, out=None, softmax_scale=None):
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        _lib.dq_decode_attention(self.k_tables, self.v_tables, q, self.k_records, self.k_mean_q,
                                 self.k_mean_scale, self.v_records, seq_lens, out, self.workspace,
                                 softmax_scale=softmax_scale, status=self.status)
        return out

    def compressed_bytes(self, tokens: int) -> int:
        """Bytes of records and key means that cover `tokens` tokens of every sequence."""
        per_tok = self.k_tables.record_bytes + self.v_tables.record_bytes
        mean = (self.head_dim + 2) * ((tokens + _lib.DQ_MEAN_WINDOW - 1) // _lib.DQ_MEAN_WINDOW)
        return self.batch * self.kv_heads * (per_tok * tokens + mean)
