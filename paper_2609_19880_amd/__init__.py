"""D-Quant hot path on MI355X: Python binding of libdq (ctypes).

The binding only marshals arguments: torch tensors are passed to the C ABI as
raw device pointers together with the current HIP stream, and every step of
the path runs in the HIP kernels of ``libdq.so``.  Importing this package
raises if the library has not been built (``__graft_entry__.build()``).

Entry points (same names as the C ABI in ``include/dq.h``):
    dq_compute_tables, dq_build_tables, dq_encode_kv,
    dq_decode_workspace_bytes, dq_decode_attention, dq_decode_attention_no_alloc,
    dq_decode_attention_partial, dq_decode_attention_merge, dq_decode_attention_residual,
    dq_decode_attention_merge_residual, dq_residual_append, dq_residual_commit,
    dq_bf16_decode_attention_partial, dq_encode_kv_paged,
    dq_decode_attention_paged_partial, dq_token_record_stride, dq_encode_kv_token,
    dq_decode_attention_token_partial, dq_fixed_bits, dq_encode_kv_fixed,
    dq_decode_attention_fixed_partial, dq_decode_symbols, dq_strerror, dq_last_error
"""

from ._lib import (  # noqa: F401
    DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_INFEASIBLE, DQ_ERR_HIP, DQ_ERR_WORKSPACE,
    DQ_STATUS_RANGE, DQ_STATUS_OVERFLOW, DQ_STATUS_CORRUPT, DQ_STATUS_WINDOW, DQ_STATUS_PAGE, DQ_MEAN_WINDOW,
    DqError, Tables, TableInfo, library_path,
    dq_compute_tables, dq_build_tables, dq_encode_kv, dq_decode_workspace_bytes,
    dq_decode_attention, dq_decode_attention_no_alloc, DQ_NO_ALLOC_SCRATCH_BYTES,
    dq_decode_attention_partial, dq_decode_attention_merge, dq_decode_attention_residual,
    dq_decode_attention_merge_residual,
    dq_residual_append, dq_residual_commit,
    dq_bf16_decode_attention_partial, dq_encode_kv_paged, dq_decode_attention_paged_partial,
    dq_token_record_stride, token_records_shape, dq_encode_kv_token, dq_decode_attention_token_partial,
    token_pool_shape, dq_encode_kv_token_paged, dq_decode_attention_token_paged_partial,
    dq_fixed_bits, dq_encode_kv_fixed, dq_decode_attention_fixed_partial,
    dq_decode_symbols, dq_strerror, dq_last_error, smallest_feasible_alpha,
)
from .cache import KVCache, StreamingKVCache, TokenKVCache  # noqa: F401
