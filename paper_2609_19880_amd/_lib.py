"""ctypes binding of libdq.so (argument marshalling only)."""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

# torch must be loaded first: libdq.so then binds to the HIP runtime torch
# ships with (same soname), so both share one runtime, device context and
# stream namespace.
import torch  # noqa: F401  (load order matters)

DQ_OK = 0
DQ_ERR_INVALID_ARG = 1
DQ_ERR_INFEASIBLE = 2
DQ_ERR_HIP = 3
DQ_ERR_WORKSPACE = 4

DQ_STATUS_RANGE = 1
DQ_STATUS_OVERFLOW = 2
DQ_STATUS_CORRUPT = 4
DQ_STATUS_WINDOW = 8
DQ_STATUS_PAGE = 16

DQ_MEAN_WINDOW = 128
LAMBDA_STEPS = 512

_HERE = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_HERE, "libdq.so")


class DqError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        detail = f" [{dq_last_error()}]" if code == DQ_ERR_HIP else ""
        super().__init__(f"{where}: {dq_strerror(code)} (code {code}){detail}")


class _Config(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("levels", ctypes.c_int32),
                ("precision_bits", ctypes.c_int32), ("record_bytes", ctypes.c_int32),
                ("alpha", ctypes.c_double), ("prerotated", ctypes.c_int32)]


class _Info(ctypes.Structure):
    _fields_ = [("record_bytes", ctypes.c_int32), ("feasible", ctypes.c_int32),
                ("cheapest", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("budget_q16", ctypes.c_int64), ("min_cost_q16", ctypes.c_int64),
                ("expected_max", ctypes.c_double)]


def _load():
    path = library_path()
    if not os.path.exists(path):
        raise ImportError(f"libdq.so is not built ({path}); run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.dq_compute_tables.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(_Info), P, P, P, P, P]
    lib.dq_compute_tables.restype = ctypes.c_int
    lib.dq_build_tables.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(P), ctypes.POINTER(_Info)]
    lib.dq_build_tables.restype = ctypes.c_int
    lib.dq_free_tables.argtypes = [P]
    lib.dq_free_tables.restype = None
    lib.dq_encode_kv.argtypes = [P, P, I64, I64, I64, I32, I32, I32, I32, I32, P, P, P, P, P]
    lib.dq_encode_kv.restype = ctypes.c_int
    lib.dq_decode_workspace_bytes.argtypes = [I32, I32, I32, I32, I32]
    lib.dq_decode_workspace_bytes.restype = SZ
    lib.dq_decode_attention.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32, ctypes.c_float,
                                        P, P, SZ, P, P]
    lib.dq_decode_attention.restype = ctypes.c_int
    lib.dq_decode_attention_no_alloc.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32, ctypes.c_float,
                                                 P, P, P]
    lib.dq_decode_attention_no_alloc.restype = ctypes.c_int
    lib.dq_decode_attention_partial.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32,
                                                ctypes.c_float, P, SZ, P, P]
    lib.dq_decode_attention_partial.restype = ctypes.c_int
    lib.dq_decode_attention_merge.argtypes = [I32, I32, I32, P, I32, P, SZ, P, P]
    lib.dq_decode_attention_merge.restype = ctypes.c_int
    lib.dq_decode_attention_residual.argtypes = [P, I32, I32, I32, P, P, P, P, I32, I32, ctypes.c_float,
                                                 P, SZ, P]
    lib.dq_decode_attention_residual.restype = ctypes.c_int
    lib.dq_decode_attention_merge_residual.argtypes = [P, I32, I32, I32, P, P, P, P, I32, I32, ctypes.c_float,
                                                       P, SZ, P, P]
    lib.dq_decode_attention_merge_residual.restype = ctypes.c_int
    lib.dq_encode_kv_paged.argtypes = [P, P, I64, I64, I64, I32, I32, I32, I32, P, I32, I32, I32, P, P, P, P, P]
    lib.dq_encode_kv_paged.restype = ctypes.c_int
    lib.dq_decode_attention_paged_partial.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32, I32, I32, P,
                                                      ctypes.c_float, P, SZ, P, P]
    lib.dq_decode_attention_paged_partial.restype = ctypes.c_int
    lib.dq_token_record_stride.argtypes = [P]
    lib.dq_token_record_stride.restype = I32
    lib.dq_encode_kv_token.argtypes = [P, P, I64, I64, I64, I32, I32, I32, I32, I32, P, P, P, P, P]
    lib.dq_encode_kv_token.restype = ctypes.c_int
    lib.dq_decode_attention_token_partial.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32, ctypes.c_float,
                                                      P, SZ, P, P]
    lib.dq_decode_attention_token_partial.restype = ctypes.c_int
    lib.dq_encode_kv_token_paged.argtypes = [P, P, I64, I64, I64, I32, I32, I32, I32, P, I32, I32, I32, P, P, P,
                                             P, P]
    lib.dq_encode_kv_token_paged.restype = ctypes.c_int
    lib.dq_decode_attention_token_paged_partial.argtypes = [P, P, P, I32, I32, I32, P, P, P, P, P, I32, I32, I32,
                                                            P, ctypes.c_float, P, SZ, P, P]
    lib.dq_decode_attention_token_paged_partial.restype = ctypes.c_int
    lib.dq_fixed_bits.argtypes = [I32, I32]
    lib.dq_fixed_bits.restype = I32
    lib.dq_encode_kv_fixed.argtypes = [I32, I32, P, I64, I64, I64, I32, I32, I32, I32, I32, P, P, P, P, P]
    lib.dq_encode_kv_fixed.restype = ctypes.c_int
    lib.dq_decode_attention_fixed_partial.argtypes = [P, I32, I32, I32, P, P, P, P, P, I32, ctypes.c_float,
                                                      P, SZ, P, P]
    lib.dq_decode_attention_fixed_partial.restype = ctypes.c_int
    lib.dq_bf16_decode_attention_partial.argtypes = [P, I32, I32, I32, P, P, P, I32, ctypes.c_float, P, SZ, P]
    lib.dq_bf16_decode_attention_partial.restype = ctypes.c_int
    lib.dq_residual_append.argtypes = [P, P, I32, I32, I32, P, P, P, P, I32, P, P]
    lib.dq_residual_append.restype = ctypes.c_int
    lib.dq_residual_commit.argtypes = [P, P, I32, I32, P, P]
    lib.dq_residual_commit.restype = ctypes.c_int
    lib.dq_decode_symbols.argtypes = [P, P, I64, P, P, P, P]
    lib.dq_decode_symbols.restype = ctypes.c_int
    lib.dq_strerror.argtypes = [ctypes.c_int]
    lib.dq_strerror.restype = ctypes.c_char_p
    lib.dq_last_error.argtypes = []
    lib.dq_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def dq_strerror(code: int) -> str:
    return _lib.dq_strerror(int(code)).decode()


def dq_last_error() -> str:
    return _lib.dq_last_error().decode()


@dataclass
class TableInfo:
    record_bytes: int
    feasible: bool
    cheapest: int
    budget_q16: int
    min_cost_q16: int
    expected_max: float


def _cfg(head_dim, levels, precision_bits, record_bytes, alpha, prerotated=False) -> _Config:
    return _Config(int(head_dim), int(levels), int(precision_bits), int(record_bytes), float(alpha),
                   1 if prerotated else 0)


def _info(i: _Info) -> TableInfo:
    return TableInfo(i.record_bytes, bool(i.feasible), i.cheapest, i.budget_q16, i.min_cost_q16,
                     i.expected_max)


def dq_compute_tables(head_dim: int, levels: int, precision_bits: int, record_bytes: int,
                      alpha: float):
    """Host-only table build.  Returns (info, dict of numpy arrays) or raises."""
    cfg = _cfg(head_dim, levels, precision_bits, record_bytes, alpha)
    info = _Info()
    M, P = int(levels), 1 << int(precision_bits)
    freq = np.zeros(M, np.int32)
    cum = np.zeros(M, np.int32)
    cost = np.zeros(M, np.int32)
    sym = np.zeros(P, np.uint8)
    lam = np.zeros(LAMBDA_STEPS, np.float32)
    rc = _lib.dq_compute_tables(ctypes.byref(cfg), ctypes.byref(info), freq.ctypes.data,
                                cum.ctypes.data, cost.ctypes.data, sym.ctypes.data, lam.ctypes.data)
    if rc not in (DQ_OK, DQ_ERR_INFEASIBLE):
        raise DqError(rc, "dq_compute_tables")
    return _info(info), {"freq": freq, "cum": cum, "cost": cost, "sym_of_z": sym, "lambda": lam}


class Tables:
    """Owner of a dq_tables handle (host + device copy on the current device)."""

    def __init__(self, head_dim: int, levels: int, precision_bits: int, record_bytes: int,
                 alpha: float, prerotated: bool = False):
        """prerotated: the tensor arrives already in the rotated basis (values
        whose rotation is folded into the projection weights): no online
        Hadamard in the encoder, and decode attention leaves the query (keys)
        or the output (values) in that basis."""
        self.head_dim = int(head_dim)
        self.levels = int(levels)
        self.precision_bits = int(precision_bits)
        self.record_bytes = int(record_bytes)
        self.alpha = float(alpha)
        self.prerotated = bool(prerotated)
        cfg = _cfg(head_dim, levels, precision_bits, record_bytes, alpha, prerotated)
        handle = ctypes.c_void_p()
        info = _Info()
        self._handle = None
        rc = _lib.dq_build_tables(ctypes.byref(cfg), ctypes.byref(handle), ctypes.byref(info))
        self.info = _info(info)
        if rc != DQ_OK:
            raise DqError(rc, "dq_build_tables")
        self._handle = handle

    @property
    def handle(self):
        return self._handle

    def __del__(self):
        h = getattr(self, "_handle", None)
        if h is not None and _lib is not None:
            _lib.dq_free_tables(h)
            self._handle = None


def dq_build_tables(head_dim: int, levels: int, precision_bits: int, record_bytes: int,
                    alpha: float, prerotated: bool = False) -> Tables:
    return Tables(head_dim, levels, precision_bits, record_bytes, alpha, prerotated)


def smallest_feasible_alpha(head_dim: int, levels: int, precision_bits: int, record_bytes: int,
                            start: float = 1.4, step: float = 0.1, stop: float = 64.0) -> float:
    """Smallest alpha on the grid start + k * step for which the table fits."""
    k = 0
    while True:
        a = round(start + k * step, 10)
        if a > stop:
            raise DqError(DQ_ERR_INFEASIBLE, "smallest_feasible_alpha")
        info, _ = dq_compute_tables(head_dim, levels, precision_bits, record_bytes, a)
        if info.feasible:
            return a
        k += 1


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _check(rc: int, where: str):
    if rc != DQ_OK:
        raise DqError(rc, where)


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def dq_encode_kv(tables: Tables, kv, t0: int, t_cap: int, records, mean_q=None, mean_scale=None,
                 status=None, stream=None):
    """Append kv (bf16 [B, T_new, H, d] on the GPU, channels contiguous) at
    cache position t0.  records: uint8 [B, H, t_cap, C]; keys also pass
    mean_q int8 [B, H, t_cap/128, d] and mean_scale int16/float16 [B, H, t_cap/128]."""
    import torch
    _need(kv.is_cuda and kv.dtype == torch.bfloat16 and kv.dim() == 4, "kv must be bf16 [B,T,H,d] on the GPU")
    B, T, H, d = kv.shape
    _need(kv.stride(3) == 1 and d == tables.head_dim, "kv channels must be contiguous and match head_dim")
    _need(records.is_cuda and records.dtype == torch.uint8 and records.is_contiguous()
          and tuple(records.shape) == (B, H, t_cap, tables.record_bytes), "records shape/dtype")
    if mean_q is not None:
        _need(mean_scale is not None, "mean_q and mean_scale go together")
        _need(mean_q.dtype == torch.int8 and mean_q.is_contiguous()
              and tuple(mean_q.shape) == (B, H, t_cap // DQ_MEAN_WINDOW, d), "mean_q shape/dtype")
        _need(mean_scale.element_size() == 2 and mean_scale.is_contiguous()
              and tuple(mean_scale.shape) == (B, H, t_cap // DQ_MEAN_WINDOW), "mean_scale shape/dtype")
    if status is not None:
        _need(status.is_cuda and status.element_size() == 4, "status must be a 4-byte device word")
    rc = _lib.dq_encode_kv(tables.handle, _ptr(kv), kv.stride(0), kv.stride(1), kv.stride(2),
                           B, H, int(t0), T, int(t_cap), _ptr(records), _ptr(mean_q), _ptr(mean_scale),
                           _ptr(status), _stream(stream))
    _check(rc, "dq_encode_kv")


def dq_decode_workspace_bytes(batch: int, q_heads: int, kv_heads: int, t_cap: int,
                              head_dim: int = 128) -> int:
    return int(_lib.dq_decode_workspace_bytes(batch, q_heads, kv_heads, t_cap, head_dim))


def _attention_args(k_tables, v_tables, q, k_records, k_mean_q, k_mean_scale, v_records, seq_lens, workspace):
    import torch
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(k_records.dim() == 4 and k_records.is_contiguous() and k_records.dtype == torch.uint8, "k_records")
    _, Hkv, t_cap, Ck = k_records.shape
    _need(Ck == k_tables.record_bytes and k_records.shape[0] == B, "k_records shape")
    _need(v_records.is_contiguous() and tuple(v_records.shape) == (B, Hkv, t_cap, v_tables.record_bytes),
          "v_records shape")
    _need(k_mean_q.is_contiguous() and tuple(k_mean_q.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW, d), "k_mean_q")
    _need(k_mean_scale.is_contiguous() and tuple(k_mean_scale.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW),
          "k_mean_scale")
    _need(seq_lens.is_cuda and seq_lens.dtype == torch.int32 and seq_lens.numel() == B, "seq_lens")
    return B, Hq, Hkv, t_cap, d, workspace.numel() * workspace.element_size()


def dq_decode_attention_partial(k_tables: Tables, v_tables: Tables, q, k_records, k_mean_q, k_mean_scale,
                                v_records, seq_lens, workspace, softmax_scale=None, status=None, stream=None):
    """First half of a decode step: per-chunk softmax partials into the workspace."""
    B, Hq, Hkv, t_cap, d, ws_bytes = _attention_args(k_tables, v_tables, q, k_records, k_mean_q,
                                                     k_mean_scale, v_records, seq_lens, workspace)
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_partial(k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv,
                                          _ptr(k_records), _ptr(k_mean_q), _ptr(k_mean_scale),
                                          _ptr(v_records), _ptr(seq_lens), t_cap, ctypes.c_float(scale),
                                          _ptr(workspace), ws_bytes, _ptr(status), _stream(stream))
    _check(rc, "dq_decode_attention_partial")


def dq_decode_attention_merge(batch: int, q_heads: int, kv_heads: int, seq_lens, t_cap: int, workspace, out,
                              stream=None):
    """Second half: log-sum-exp merge of the chunk partials into out fp32 [B, Hq, d]."""
    import torch
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous()
          and tuple(out.shape) == (batch, q_heads, 128), "out")
    ws_bytes = workspace.numel() * workspace.element_size()
    rc = _lib.dq_decode_attention_merge(batch, q_heads, kv_heads, _ptr(seq_lens), t_cap, _ptr(workspace),
                                        ws_bytes, _ptr(out), _stream(stream))
    _check(rc, "dq_decode_attention_merge")


def _ring_args(res_k, res_v, seq_lens, res_lens):
    import torch
    _need(res_k.is_cuda and res_k.dtype == torch.bfloat16 and res_k.is_contiguous() and res_k.dim() == 4,
          "res_k must be bf16 [B, Hkv, r_cap, d]")
    _need(res_v.is_cuda and res_v.dtype == torch.bfloat16 and res_v.is_contiguous()
          and res_v.shape == res_k.shape, "res_v must match res_k")
    B = res_k.shape[0]
    for t, name in ((seq_lens, "seq_lens"), (res_lens, "res_lens")):
        _need(t.is_cuda and t.dtype == torch.int32 and t.is_contiguous() and t.numel() == B, name)
    return res_k.shape


def dq_decode_attention_residual(q, res_k, res_v, seq_lens, res_lens, t_cap: int, workspace,
                                 softmax_scale=None, stream=None):
    """Residual window's partial: between dq_decode_attention_partial and _merge."""
    import torch
    B, Hkv, r_cap, d = _ring_args(res_k, res_v, seq_lens, res_lens)
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3
          and q.shape[0] == B and q.shape[2] == d, "q")
    Hq = q.shape[1]
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_residual(_ptr(q), B, Hq, Hkv, _ptr(res_k), _ptr(res_v), _ptr(seq_lens),
                                           _ptr(res_lens), r_cap, int(t_cap), ctypes.c_float(scale),
                                           _ptr(workspace), workspace.numel() * workspace.element_size(),
                                           _stream(stream))
    _check(rc, "dq_decode_attention_residual")


def dq_decode_attention_merge_residual(q, res_k, res_v, seq_lens, res_lens, t_cap: int, workspace, out,
                                       softmax_scale=None, stream=None):
    """Residual window and merge in one launch: after any _partial call, writes
    out fp32 [B, Hq, d] as dq_decode_attention_residual + _merge would."""
    import torch
    B, Hkv, r_cap, d = _ring_args(res_k, res_v, seq_lens, res_lens)
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3
          and q.shape[0] == B and q.shape[2] == d, "q")
    Hq = q.shape[1]
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous()
          and tuple(out.shape) == (B, Hq, 128), "out")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_merge_residual(_ptr(q), B, Hq, Hkv, _ptr(res_k), _ptr(res_v), _ptr(seq_lens),
                                                 _ptr(res_lens), r_cap, int(t_cap), ctypes.c_float(scale),
                                                 _ptr(workspace), workspace.numel() * workspace.element_size(),
                                                 _ptr(out), _stream(stream))
    _check(rc, "dq_decode_attention_merge_residual")


def _pool_args(tables, record_pool, block_table, mean_q_pool=None, mean_scale_pool=None):
    import torch
    _need(record_pool.is_cuda and record_pool.dtype == torch.uint8 and record_pool.is_contiguous()
          and record_pool.dim() == 4 and record_pool.shape[3] == tables.record_bytes, "record pool")
    num_pages, H, page, _ = record_pool.shape
    _need(block_table.is_cuda and block_table.dtype == torch.int32 and block_table.is_contiguous()
          and block_table.dim() == 2, "block_table must be int32 [batch, max_pages]")
    if mean_q_pool is not None:
        _need(mean_q_pool.dtype == torch.int8 and mean_q_pool.is_contiguous()
              and tuple(mean_q_pool.shape) == (num_pages, H, page // DQ_MEAN_WINDOW, tables.head_dim), "mean_q pool")
        _need(mean_scale_pool is not None and mean_scale_pool.element_size() == 2 and mean_scale_pool.is_contiguous()
              and tuple(mean_scale_pool.shape) == (num_pages, H, page // DQ_MEAN_WINDOW), "mean_scale pool")
    return num_pages, H, page, block_table.shape[1]


def dq_encode_kv_paged(tables: Tables, kv, t0: int, block_table, record_pool, mean_q_pool=None,
                       mean_scale_pool=None, status=None, stream=None):
    """dq_encode_kv into a paged pool: record_pool uint8 [num_pages, H, page, C];
    block_table int32 [B, max_pages]; keys also pass the mean pools."""
    import torch
    _need(kv.is_cuda and kv.dtype == torch.bfloat16 and kv.dim() == 4 and kv.stride(3) == 1, "kv")
    B, T, H, d = kv.shape
    num_pages, Hp, page, max_pages = _pool_args(tables, record_pool, block_table, mean_q_pool, mean_scale_pool)
    _need(Hp == H and block_table.shape[0] == B and d == tables.head_dim, "pool/kv shapes")
    rc = _lib.dq_encode_kv_paged(tables.handle, _ptr(kv), kv.stride(0), kv.stride(1), kv.stride(2), B, H,
                                 int(t0), T, _ptr(block_table), max_pages, page, num_pages, _ptr(record_pool),
                                 _ptr(mean_q_pool), _ptr(mean_scale_pool), _ptr(status), _stream(stream))
    _check(rc, "dq_encode_kv_paged")


def dq_decode_attention_paged_partial(k_tables: Tables, v_tables: Tables, q, k_pool, mean_q_pool, mean_scale_pool,
                                      v_pool, block_table, seq_lens, workspace, softmax_scale=None, status=None,
                                      stream=None):
    """dq_decode_attention_partial over paged pools; finish with
    dq_decode_attention_merge(..., t_cap = max_pages * page_tokens, ...)."""
    import torch
    num_pages, Hkv, page, max_pages = _pool_args(k_tables, k_pool, block_table, mean_q_pool, mean_scale_pool)
    _need(v_pool.is_cuda and v_pool.dtype == torch.uint8 and v_pool.is_contiguous()
          and tuple(v_pool.shape) == (num_pages, Hkv, page, v_tables.record_bytes), "v pool")
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(block_table.shape[0] == B and seq_lens.is_cuda and seq_lens.dtype == torch.int32
          and seq_lens.numel() == B, "block_table / seq_lens")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_paged_partial(k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv, _ptr(k_pool),
                                                _ptr(mean_q_pool), _ptr(mean_scale_pool), _ptr(v_pool),
                                                _ptr(block_table), max_pages, page, num_pages, _ptr(seq_lens),
                                                ctypes.c_float(scale), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(), _ptr(status),
                                                _stream(stream))
    _check(rc, "dq_decode_attention_paged_partial")


def dq_token_record_stride(tables: Tables) -> int:
    """Bytes of a per-token record slot (C rounded up to 16)."""
    return int(_lib.dq_token_record_stride(tables.handle))


def token_records_shape(tables: Tables, batch: int, t_cap: int):
    """Shape of a per-token record buffer: [B, t_cap / 64, S / 8, 64, 8] --
    64-token tiles, 8-byte chunks outermost; token t's record is
    records[b, t // 64, :, t % 64, :] flattened (its first C bytes)."""
    S = dq_token_record_stride(tables)
    return (batch, t_cap // 64, S // 8, 64, 8)


def dq_encode_kv_token(tables: Tables, kv, t0: int, t_cap: int, records, mean_q=None, mean_scale=None,
                       status=None, stream=None):
    """Append kv (bf16 [B, T_new, H, 128] on the GPU) at cache position t0 as
    one stream per token over the H heads (tables built with head_dim 128 H).
    records: uint8 of token_records_shape(tables, B, t_cap); keys also pass
    mean_q int8 [B, H, t_cap/128, 128] and mean_scale [B, H, t_cap/128]."""
    import torch
    _need(kv.is_cuda and kv.dtype == torch.bfloat16 and kv.dim() == 4 and kv.stride(3) == 1, "kv")
    B, T, H, d = kv.shape
    _need(d == 128 and tables.head_dim == 128 * H, "per-token streams need head_dim 128 and n = 128 H")
    _need(records.is_cuda and records.dtype == torch.uint8 and records.is_contiguous()
          and tuple(records.shape) == token_records_shape(tables, B, t_cap), "records shape/dtype")
    if mean_q is not None:
        _need(mean_scale is not None, "mean_q and mean_scale go together")
        _need(mean_q.dtype == torch.int8 and mean_q.is_contiguous()
              and tuple(mean_q.shape) == (B, H, t_cap // DQ_MEAN_WINDOW, d), "mean_q shape/dtype")
        _need(mean_scale.element_size() == 2 and mean_scale.is_contiguous()
              and tuple(mean_scale.shape) == (B, H, t_cap // DQ_MEAN_WINDOW), "mean_scale shape/dtype")
    rc = _lib.dq_encode_kv_token(tables.handle, _ptr(kv), kv.stride(0), kv.stride(1), kv.stride(2), B, H,
                                 int(t0), T, int(t_cap), _ptr(records), _ptr(mean_q), _ptr(mean_scale),
                                 _ptr(status), _stream(stream))
    _check(rc, "dq_encode_kv_token")


def dq_decode_attention_token_partial(k_tables: Tables, v_tables: Tables, q, k_records, mean_q, mean_scale,
                                      v_records, seq_lens, workspace, softmax_scale=None, status=None,
                                      stream=None):
    """Split-K partials of one decode step over per-token records (shape
    token_records_shape); finish with dq_decode_attention_merge."""
    import torch
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(k_records.dim() == 5 and k_records.shape[0] == B and k_records.is_contiguous(), "k_records")
    t_cap = k_records.shape[1] * 64
    _need(tuple(k_records.shape) == token_records_shape(k_tables, B, t_cap), "k_records shape")
    Hkv = k_tables.head_dim // 128
    _need(tuple(v_records.shape) == token_records_shape(v_tables, B, t_cap) and v_records.is_contiguous(),
          "v_records")
    _need(tuple(mean_q.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW, 128) and mean_q.is_contiguous(), "mean_q")
    _need(tuple(mean_scale.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW) and mean_scale.is_contiguous(), "mean_scale")
    _need(seq_lens.is_cuda and seq_lens.dtype == torch.int32 and seq_lens.numel() == B, "seq_lens")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_token_partial(k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv,
                                                _ptr(k_records), _ptr(mean_q), _ptr(mean_scale), _ptr(v_records),
                                                _ptr(seq_lens), t_cap, ctypes.c_float(scale), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(), _ptr(status),
                                                _stream(stream))
    _check(rc, "dq_decode_attention_token_partial")


def token_pool_shape(tables: Tables, num_pages: int, page_tokens: int):
    """Shape of a paged per-token record pool: [num_pages, page / 64, S / 8, 64,
    8] -- each page holds the 64-token tiles of page_tokens tokens."""
    S = dq_token_record_stride(tables)
    return (num_pages, page_tokens // 64, S // 8, 64, 8)


def _token_pool_args(tables, record_pool, block_table, kv_heads, mean_q_pool=None, mean_scale_pool=None):
    import torch
    _need(record_pool.is_cuda and record_pool.dtype == torch.uint8 and record_pool.is_contiguous()
          and record_pool.dim() == 5, "record pool must be uint8 [num_pages, page/64, S/8, 64, 8]")
    num_pages, page = record_pool.shape[0], record_pool.shape[1] * 64
    _need(tuple(record_pool.shape) == token_pool_shape(tables, num_pages, page), "record pool shape")
    _need(block_table.is_cuda and block_table.dtype == torch.int32 and block_table.is_contiguous()
          and block_table.dim() == 2, "block_table must be int32 [batch, max_pages]")
    if mean_q_pool is not None:
        _need(mean_q_pool.dtype == torch.int8 and mean_q_pool.is_contiguous()
              and tuple(mean_q_pool.shape) == (num_pages, kv_heads, page // DQ_MEAN_WINDOW, 128), "mean_q pool")
        _need(mean_scale_pool is not None and mean_scale_pool.element_size() == 2 and mean_scale_pool.is_contiguous()
              and tuple(mean_scale_pool.shape) == (num_pages, kv_heads, page // DQ_MEAN_WINDOW), "mean_scale pool")
    return num_pages, page, block_table.shape[1]


def dq_encode_kv_token_paged(tables: Tables, kv, t0: int, block_table, record_pool, mean_q_pool=None,
                             mean_scale_pool=None, status=None, stream=None):
    """dq_encode_kv_token into a paged pool of token_pool_shape; block_table
    int32 [B, max_pages]; keys also pass the mean pools [num_pages, H, page/128, ...]."""
    import torch
    _need(kv.is_cuda and kv.dtype == torch.bfloat16 and kv.dim() == 4 and kv.stride(3) == 1, "kv")
    B, T, H, d = kv.shape
    _need(d == 128 and tables.head_dim == 128 * H, "per-token streams need head_dim 128 and n = 128 H")
    num_pages, page, max_pages = _token_pool_args(tables, record_pool, block_table, H, mean_q_pool, mean_scale_pool)
    _need(block_table.shape[0] == B, "block_table rows")
    rc = _lib.dq_encode_kv_token_paged(tables.handle, _ptr(kv), kv.stride(0), kv.stride(1), kv.stride(2), B, H,
                                       int(t0), T, _ptr(block_table), max_pages, page, num_pages, _ptr(record_pool),
                                       _ptr(mean_q_pool), _ptr(mean_scale_pool), _ptr(status), _stream(stream))
    _check(rc, "dq_encode_kv_token_paged")


def dq_decode_attention_token_paged_partial(k_tables: Tables, v_tables: Tables, q, k_pool, mean_q_pool,
                                            mean_scale_pool, v_pool, block_table, seq_lens, workspace,
                                            softmax_scale=None, status=None, stream=None):
    """dq_decode_attention_token_partial over paged pools; finish with
    dq_decode_attention_merge(..., t_cap = max_pages * page_tokens, ...)."""
    import torch
    _need(mean_q_pool is not None and mean_q_pool.dim() == 4, "mean_q pool")
    Hkv = mean_q_pool.shape[1]
    num_pages, page, max_pages = _token_pool_args(k_tables, k_pool, block_table, Hkv, mean_q_pool, mean_scale_pool)
    _need(v_pool.is_cuda and v_pool.dtype == torch.uint8 and v_pool.is_contiguous()
          and tuple(v_pool.shape) == token_pool_shape(v_tables, num_pages, page), "v pool")
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(block_table.shape[0] == B and seq_lens.is_cuda and seq_lens.dtype == torch.int32
          and seq_lens.numel() == B, "block_table / seq_lens")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_token_paged_partial(
        k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv, _ptr(k_pool), _ptr(mean_q_pool),
        _ptr(mean_scale_pool), _ptr(v_pool), _ptr(block_table), max_pages, page, num_pages, _ptr(seq_lens),
        ctypes.c_float(scale), _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(status),
        _stream(stream))
    _check(rc, "dq_decode_attention_token_paged_partial")


def dq_fixed_bits(head_dim: int, record_bytes: int) -> int:
    """Bits per symbol of the fixed-width comparator (0: no valid width)."""
    return int(_lib.dq_fixed_bits(int(head_dim), int(record_bytes)))


def dq_encode_kv_fixed(head_dim: int, record_bytes: int, kv, t0: int, t_cap: int, records, mean_q=None,
                       mean_scale=None, status=None, stream=None):
    """Fixed-width comparator encoder (App. B): kv bf16 [B, T_new, H, d] at cache
    position t0 into records uint8 [B, H, t_cap, C]; keys also pass the means."""
    import torch
    _need(kv.is_cuda and kv.dtype == torch.bfloat16 and kv.dim() == 4 and kv.stride(3) == 1, "kv")
    B, T, H, d = kv.shape
    _need(d == head_dim, "kv head_dim")
    _need(records.is_cuda and records.dtype == torch.uint8 and records.is_contiguous()
          and tuple(records.shape) == (B, H, t_cap, record_bytes), "records shape/dtype")
    if mean_q is not None:
        _need(mean_scale is not None and tuple(mean_q.shape) == (B, H, t_cap // DQ_MEAN_WINDOW, d)
              and mean_q.is_contiguous() and mean_scale.is_contiguous(), "mean buffers")
    rc = _lib.dq_encode_kv_fixed(int(head_dim), int(record_bytes), _ptr(kv), kv.stride(0), kv.stride(1),
                                 kv.stride(2), B, H, int(t0), T, int(t_cap), _ptr(records), _ptr(mean_q),
                                 _ptr(mean_scale), _ptr(status), _stream(stream))
    _check(rc, "dq_encode_kv_fixed")


def dq_decode_attention_fixed_partial(q, k_records, mean_q, mean_scale, v_records, seq_lens, workspace,
                                      softmax_scale=None, status=None, stream=None):
    """Split-K partials of one decode step over 36-byte fixed-width records
    [B, H_kv, t_cap, 36]; finish with dq_decode_attention_merge."""
    import torch
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(k_records.dim() == 4 and k_records.shape[0] == B and k_records.shape[3] == 36
          and k_records.is_contiguous() and tuple(v_records.shape) == tuple(k_records.shape)
          and v_records.is_contiguous(), "records")
    Hkv, t_cap = k_records.shape[1], k_records.shape[2]
    _need(tuple(mean_q.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW, 128) and mean_q.is_contiguous()
          and tuple(mean_scale.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW) and mean_scale.is_contiguous(), "means")
    _need(seq_lens.is_cuda and seq_lens.dtype == torch.int32 and seq_lens.numel() == B, "seq_lens")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_fixed_partial(_ptr(q), B, Hq, Hkv, _ptr(k_records), _ptr(mean_q),
                                                _ptr(mean_scale), _ptr(v_records), _ptr(seq_lens), t_cap,
                                                ctypes.c_float(scale), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(), _ptr(status),
                                                _stream(stream))
    _check(rc, "dq_decode_attention_fixed_partial")


def dq_bf16_decode_attention_partial(q, k, v, seq_lens, workspace, softmax_scale=None, stream=None):
    """Comparator: split-K partials of plain BF16 attention over k, v bf16
    [B, Hkv, t_cap, d]; finish with dq_decode_attention_merge."""
    import torch
    for t, name in ((k, "k"), (v, "v")):
        _need(t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and t.dim() == 4, name)
    _need(v.shape == k.shape, "v must match k")
    B, Hkv, t_cap, d = k.shape
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3
          and q.shape[0] == B and q.shape[2] == d, "q")
    _need(seq_lens.is_cuda and seq_lens.dtype == torch.int32 and seq_lens.numel() == B, "seq_lens")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_bf16_decode_attention_partial(_ptr(q), B, q.shape[1], Hkv, _ptr(k), _ptr(v), _ptr(seq_lens),
                                               t_cap, ctypes.c_float(scale), _ptr(workspace),
                                               workspace.numel() * workspace.element_size(), _stream(stream))
    _check(rc, "dq_bf16_decode_attention_partial")


def dq_residual_append(k_new, v_new, res_k, res_v, seq_lens, res_lens, status=None, stream=None):
    """One token per sequence (bf16 [B, Hkv, d]) into the residual ring."""
    import torch
    B, Hkv, r_cap, d = _ring_args(res_k, res_v, seq_lens, res_lens)
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        _need(t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and tuple(t.shape) == (B, Hkv, d),
              name)
    rc = _lib.dq_residual_append(_ptr(k_new), _ptr(v_new), B, Hkv, d, _ptr(res_k), _ptr(res_v), _ptr(seq_lens),
                                 _ptr(res_lens), r_cap, _ptr(status), _stream(stream))
    _check(rc, "dq_residual_append")


def dq_residual_commit(seq_lens, res_lens, n: int, status=None, stream=None):
    """The oldest n residual tokens were encoded: move them to the compressed side."""
    rc = _lib.dq_residual_commit(_ptr(seq_lens), _ptr(res_lens), seq_lens.numel(), int(n), _ptr(status),
                                 _stream(stream))
    _check(rc, "dq_residual_commit")


def dq_decode_attention(k_tables: Tables, v_tables: Tables, q, k_records, k_mean_q, k_mean_scale,
                        v_records, seq_lens, out, workspace, softmax_scale=None, status=None,
                        stream=None):
    """One decode step: q bf16 [B, Hq, d] -> out fp32 [B, Hq, d]."""
    import torch
    B, Hq, Hkv, t_cap, d, ws_bytes = _attention_args(k_tables, v_tables, q, k_records, k_mean_q,
                                                     k_mean_scale, v_records, seq_lens, workspace)
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and tuple(out.shape) == (B, Hq, d),
          "out")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention(k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv,
                                  _ptr(k_records), _ptr(k_mean_q), _ptr(k_mean_scale), _ptr(v_records),
                                  _ptr(seq_lens), t_cap, ctypes.c_float(scale), _ptr(out),
                                  _ptr(workspace), ws_bytes, _ptr(status), _stream(stream))
    _check(rc, "dq_decode_attention")


DQ_NO_ALLOC_SCRATCH_BYTES = 8 << 20


def dq_decode_attention_no_alloc(k_tables: Tables, v_tables: Tables, q, k_records, k_mean_q, k_mean_scale,
                                 v_records, seq_lens, out, softmax_scale=None, status=None, stream=None):
    """dq_decode_attention with the split-K workspace in the library's static
    per-device scratch array: nothing is allocated.  Calls that overlap on one
    device race (they share the array)."""
    import torch
    _need(q.is_cuda and q.dtype == torch.bfloat16 and q.is_contiguous() and q.dim() == 3, "q")
    B, Hq, d = q.shape
    _need(k_records.dim() == 4 and k_records.is_contiguous() and k_records.dtype == torch.uint8, "k_records")
    _, Hkv, t_cap, Ck = k_records.shape
    _need(Ck == k_tables.record_bytes and k_records.shape[0] == B, "k_records shape")
    _need(v_records.is_contiguous() and tuple(v_records.shape) == (B, Hkv, t_cap, v_tables.record_bytes),
          "v_records shape")
    _need(k_mean_q.is_contiguous() and tuple(k_mean_q.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW, d), "k_mean_q")
    _need(k_mean_scale.is_contiguous() and tuple(k_mean_scale.shape) == (B, Hkv, t_cap // DQ_MEAN_WINDOW),
          "k_mean_scale")
    _need(seq_lens.is_cuda and seq_lens.dtype == torch.int32 and seq_lens.numel() == B, "seq_lens")
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and tuple(out.shape) == (B, Hq, d),
          "out")
    scale = (1.0 / d ** 0.5) if softmax_scale is None else float(softmax_scale)
    rc = _lib.dq_decode_attention_no_alloc(k_tables.handle, v_tables.handle, _ptr(q), B, Hq, Hkv,
                                           _ptr(k_records), _ptr(k_mean_q), _ptr(k_mean_scale), _ptr(v_records),
                                           _ptr(seq_lens), t_cap, ctypes.c_float(scale), _ptr(out), _ptr(status),
                                           _stream(stream))
    _check(rc, "dq_decode_attention_no_alloc")


def dq_decode_symbols(tables: Tables, records, sym, header=None, status=None, stream=None):
    """records uint8 [..., C] -> sym uint8 [..., d] (+ header int16 [..., 2])."""
    import torch
    _need(records.is_contiguous() and records.dtype == torch.uint8 and records.shape[-1] == tables.record_bytes,
          "records")
    S = records.numel() // tables.record_bytes
    _need(sym.is_contiguous() and sym.dtype == torch.uint8 and sym.numel() == S * tables.head_dim, "sym")
    if header is not None:
        _need(header.is_contiguous() and header.element_size() == 2 and header.numel() == 2 * S, "header")
    rc = _lib.dq_decode_symbols(tables.handle, _ptr(records), S, _ptr(sym), _ptr(header), _ptr(status),
                                _stream(stream))
    _check(rc, "dq_decode_symbols")
