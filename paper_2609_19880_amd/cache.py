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

    def partial(self, q, seq_lens, softmax_scale=None):
        """Split-K partials of one decode step into the workspace (finish with merge)."""
        _lib.dq_decode_attention_partial(self.k_tables, self.v_tables, q, self.k_records, self.k_mean_q,
                                         self.k_mean_scale, self.v_records, seq_lens, self.workspace,
                                         softmax_scale=softmax_scale, status=self.status)

    def merge(self, seq_lens, out):
        _lib.dq_decode_attention_merge(self.batch, self.q_heads, self.kv_heads, seq_lens, self.t_cap,
                                       self.workspace, out)

    def compressed_bytes(self, tokens: int) -> int:
        """Bytes of records and key means that cover `tokens` tokens of every sequence."""
        per_tok = self.k_tables.record_bytes + self.v_tables.record_bytes
        mean = (self.head_dim + 2) * ((tokens + _lib.DQ_MEAN_WINDOW - 1) // _lib.DQ_MEAN_WINDOW)
        return self.batch * self.kv_heads * (per_tok * tokens + mean)


class TokenKVCache:
    """Compressed cache with one stream per token over all KV heads (tables
    built with head_dim 128 kv_heads): records of token_records_shape per
    tensor (64-token tiles, 8-byte chunks outermost), key means per head as in
    KVCache."""

    def __init__(self, batch: int, kv_heads: int, q_heads: int, t_cap: int, k_tables, v_tables,
                 device="cuda"):
        if t_cap % _lib.DQ_MEAN_WINDOW:
            raise ValueError("t_cap must be a multiple of 128")
        if k_tables.head_dim != 128 * kv_heads or v_tables.head_dim != 128 * kv_heads:
            raise ValueError("per-token tables need head_dim = 128 kv_heads")
        d = 128
        self.batch, self.kv_heads, self.q_heads, self.t_cap, self.head_dim = batch, kv_heads, q_heads, t_cap, d
        self.k_tables, self.v_tables = k_tables, v_tables
        nw = t_cap // _lib.DQ_MEAN_WINDOW
        self.k_records = torch.zeros(_lib.token_records_shape(k_tables, batch, t_cap), dtype=torch.uint8,
                                     device=device)
        self.v_records = torch.zeros(_lib.token_records_shape(v_tables, batch, t_cap), dtype=torch.uint8,
                                     device=device)
        self.k_mean_q = torch.zeros((batch, kv_heads, nw, d), dtype=torch.int8, device=device)
        self.k_mean_scale = torch.zeros((batch, kv_heads, nw), dtype=torch.int16, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.workspace = torch.empty(
            _lib.dq_decode_workspace_bytes(batch, q_heads, kv_heads, t_cap, d), dtype=torch.uint8, device=device)

    def append(self, k, v, t0: int):
        """Encode bf16 k, v [B, T_new, H, 128] as cache tokens [t0, t0 + T_new)."""
        _lib.dq_encode_kv_token(self.k_tables, k, t0, self.t_cap, self.k_records, self.k_mean_q,
                                self.k_mean_scale, self.status)
        _lib.dq_encode_kv_token(self.v_tables, v, t0, self.t_cap, self.v_records, None, None, self.status)

    def partial(self, q, seq_lens, softmax_scale=None):
        _lib.dq_decode_attention_token_partial(self.k_tables, self.v_tables, q, self.k_records, self.k_mean_q,
                                               self.k_mean_scale, self.v_records, seq_lens, self.workspace,
                                               softmax_scale=softmax_scale, status=self.status)

    def merge(self, seq_lens, out):
        _lib.dq_decode_attention_merge(self.batch, self.q_heads, self.kv_heads, seq_lens, self.t_cap,
                                       self.workspace, out)

    def attend(self, q, seq_lens, out=None, softmax_scale=None):
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        self.partial(q, seq_lens, softmax_scale)
        self.merge(seq_lens, out)
        return out


class StreamingKVCache:
    """A compressed cache plus the BF16 residual window of the newest tokens.

    Sec. 5.1 keeps the most recent tokens in BF16.  Here the newest tokens of
    every sequence sit raw in a ring of 2 x 128 slots (the library's residual
    window); when the ring is full its oldest 128 tokens are encoded as one
    key-mean window and leave it, so at least the 128 most recent tokens are
    always raw.  Decode attention runs over both parts in one step.  All
    sequences of the batch advance together (same length).

    streams="head" keeps one stream per (token, KV head) (a KVCache);
    streams="token" the paper's default grouping, one stream per token over
    all KV heads (a TokenKVCache, tables built with head_dim 128 kv_heads).
    The ring, its append and commit, and the residual attention are the same
    for both.
    """

    WINDOW = _lib.DQ_MEAN_WINDOW

    def __init__(self, batch: int, kv_heads: int, q_heads: int, t_cap: int, k_tables, v_tables,
                 device="cuda", r_cap: int = 256, streams: str = "head"):
        if r_cap % self.WINDOW or not (2 * self.WINDOW <= r_cap <= 256):
            raise ValueError("r_cap must be 256 (two mean windows)")
        if streams == "head":
            self.cache = KVCache(batch, kv_heads, q_heads, t_cap, k_tables, v_tables, device=device)
        elif streams == "token":
            self.cache = TokenKVCache(batch, kv_heads, q_heads, t_cap, k_tables, v_tables, device=device)
        else:
            raise ValueError("streams must be 'head' or 'token'")
        self.streams = streams
        d = self.cache.head_dim
        self.r_cap = r_cap
        self.res_k = torch.zeros((batch, kv_heads, r_cap, d), dtype=torch.bfloat16, device=device)
        self.res_v = torch.zeros_like(self.res_k)
        self.seq_lens = torch.zeros(batch, dtype=torch.int32, device=device)   # compressed tokens
        self.res_lens = torch.zeros(batch, dtype=torch.int32, device=device)   # residual tokens
        self.n_comp = 0
        self.n_res = 0

    @property
    def status(self):
        return self.cache.status

    def __len__(self) -> int:
        return self.n_comp + self.n_res

    def prefill(self, k, v):
        """k, v bf16 [B, T, H, d] into an empty cache: whole windows are encoded,
        the last 128..255 tokens (all of them if T < 128) stay raw."""
        if len(self):
            raise RuntimeError("prefill needs an empty cache")
        T = k.shape[1]
        n_enc = max(0, (T - self.WINDOW) // self.WINDOW * self.WINDOW)
        if n_enc:
            self.cache.append(k[:, :n_enc], v[:, :n_enc], 0)
            self.seq_lens += n_enc
            self.n_comp = n_enc
        for t in range(n_enc, T):
            self.append(k[:, t].contiguous(), v[:, t].contiguous())

    def append(self, k1, v1):
        """One decode token per sequence: k1, v1 bf16 [B, H, d]."""
        if self.n_res == self.r_cap:
            self._flush()
        _lib.dq_residual_append(k1, v1, self.res_k, self.res_v, self.seq_lens, self.res_lens, self.status)
        self.n_res += 1
        if self.n_res == self.r_cap:
            self._flush()

    def _flush(self):
        W = self.WINDOW
        if self.n_comp + W > self.cache.t_cap:
            raise RuntimeError("compressed cache is full")
        s = self.n_comp % self.r_cap
        k = self.res_k[:, :, s:s + W].permute(0, 2, 1, 3)     # [B, W, H, d] view of the ring
        v = self.res_v[:, :, s:s + W].permute(0, 2, 1, 3)
        self.cache.append(k, v, self.n_comp)
        _lib.dq_residual_commit(self.seq_lens, self.res_lens, W, self.status)
        self.n_comp += W
        self.n_res -= W

    def attend(self, q, out=None, softmax_scale=None):
        """q bf16 [B, Hq, d] -> out fp32 [B, Hq, d] over every token so far."""
        c = self.cache
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        c.partial(q, self.seq_lens, softmax_scale)
        _lib.dq_decode_attention_merge_residual(q, self.res_k, self.res_v, self.seq_lens, self.res_lens, c.t_cap,
                                                c.workspace, out, softmax_scale=softmax_scale)
        return out
