/*
 * dq.h -- C ABI of the D-Quant hot path on MI355X (gfx950).
 *
 * D-Quant (arXiv 2609.19880) stores each token's key or value vector as a
 * fixed-size record: Hadamard rotation, (keys) windowed channel-mean removal,
 * a token-wise min-max affine grid with M levels, a rate-constrained
 * assignment ("drift") that makes the entropy-coded length fit the record,
 * and rANS with a static table derived from standard-normal CDF mass
 * (Sec. 4, Alg. 1).  Decode attention reads the records at fixed stride,
 * rANS-decodes them (Alg. 2) and attends with the affine folded into the
 * contractions (App. A, Eq. fold-key / fold-value).
 *
 * One stream is one (token, KV head): n = head_dim values.  A record of C
 * bytes is laid out as
 *     [scale fp16 LE][offset fp16 LE][rANS state u32 LE][renorm bytes, in the
 *     order the decoder reads them][zero padding]
 * so its rANS budget (Eq. budget) is B = 8 (C - 4) - 32 bits.  The rANS state
 * lives in [2^21, 2^29) and is renormalized one byte at a time.
 *
 * Conventions for every call:
 *  - Device pointers are plain device addresses on the device that was current
 *    when the tables were built; the caller owns every device buffer.
 *  - Work is enqueued on `stream` (a hipStream_t, NULL = the null stream) and
 *    is asynchronous: no call synchronizes, and device-side errors are reported
 *    through the caller's `status` word (see DQ_STATUS_*), readable once the
 *    stream has finished.
 *  - Host-side validation failures return an error code before anything is
 *    enqueued.  No C++ exception crosses this interface.
 *  - bf16 and fp16 values are passed as their 16-bit patterns.
 */
#ifndef DQ_H
#define DQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define DQ_OK 0
#define DQ_ERR_INVALID_ARG 1 /* a size, pointer or layout is out of range    */
#define DQ_ERR_INFEASIBLE 2  /* n * min cost exceeds the budget (Tab. 2 "--") */
#define DQ_ERR_HIP 3         /* a HIP runtime call or a launch failed          */
#define DQ_ERR_WORKSPACE 4   /* the workspace is missing or too small          */

/* Bits OR-ed into the caller's device status word. */
#define DQ_STATUS_RANGE 1u    /* encode: non-finite input, or scale/offset/mean overflowed fp16 */
#define DQ_STATUS_OVERFLOW 2u /* encode: a stream could not be fitted into its record (written as
                                 zeros); the coded-length bound makes this unreachable for n <= 1024 */
#define DQ_STATUS_CORRUPT 4u  /* decode: a record did not end in state 2^21 inside its C bytes  */
#define DQ_STATUS_WINDOW 8u   /* residual window: append to a full ring, or commit more than it holds */
#define DQ_STATUS_PAGE 16u    /* paged layout: a block-table entry outside the page pool (skipped)     */

/* Fixed parameters of the format. */
#define DQ_MEAN_WINDOW 128 /* tokens per key-mean window (windows start at token 0) */
#define DQ_MAX_LEVELS 64

/*
 * Coding parameters of one tensor (keys or values).  The per-token bit budget
 * is given as the record size: bits per element = 8 * record_bytes / head_dim
 * (Sec. 4.2 Eq. budget; Sec. 4.4 lets keys and values differ).
 */
typedef struct dq_config {
    int32_t head_dim;       /* n: values per stream, a power of 2 in 64..1024;
                               encode takes n <= 256, decode attention n = 128 */
    int32_t levels;         /* M: quantization levels, 2..64 (Eq. affine_token) */
    int32_t precision_bits; /* p: rANS precision, 8..12 (Eq. rans)              */
    int32_t record_bytes;   /* C: record size in bytes, 9..2n+8                 */
    double alpha;           /* sharpening exponent, >= 1 (Sec. 4.4; paper 1.4)  */
    int32_t prerotated;     /* 0: the library rotates every head's vector with
                               the Hadamard matrix (Sec. 4.2; keys need this,
                               RoPE does not commute with it).  1: the tensor
                               arrives already in the rotated basis, as values
                               do when the rotation is folded into the
                               projection weights offline (Sec. 4.2): no
                               online rotation, see dq_decode_attention.     */
} dq_config;

typedef struct dq_table_info {
    int32_t record_bytes;   /* C                                                 */
    int32_t feasible;       /* 1 if n * min_cost_q16 <= budget_q16               */
    int32_t cheapest;       /* lowest-index symbol of minimum cost               */
    int32_t reserved;
    int64_t budget_q16;     /* B = (8 (C - 4) - 32) * 2^16                       */
    int64_t min_cost_q16;   /* n * min_m R_m                                     */
    double expected_max;    /* a_n = E[max of n standard normals]                */
} dq_table_info;

/* Opaque coding tables: host copy plus a device copy, immutable once built. */
typedef struct dq_tables dq_tables;

/*
 * Builds the entropy model on the host only (no GPU needed):
 * level probabilities from normal CDF mass on the grid [-a_n, a_n] (the
 * order-statistics model of normal samples, Sec. 4.2), sharpened p^alpha
 * (Sec. 4.4), apportioned to integers summing to 2^p (Eq. rans), Q16 costs R_m = round(2^16 (p - log2 f_m))
 * (Alg. 1), the lambda grid 2^(k/512) as fp32, and the feasibility test.
 * Output arrays may be NULL; sizes: freq, cum, cost_q16: levels entries;
 * sym_of_z: 2^p entries; lambda512: 512 entries.
 * Returns DQ_OK, DQ_ERR_INVALID_ARG, or DQ_ERR_INFEASIBLE (info is filled).
 */
int dq_compute_tables(const dq_config* cfg, dq_table_info* info, int32_t* freq,
                      int32_t* cum, int32_t* cost_q16, uint8_t* sym_of_z,
                      float* lambda512);

/*
 * Same tables, copied to the current HIP device.  On DQ_OK *out owns host and
 * device memory until dq_free_tables.  An infeasible configuration returns
 * DQ_ERR_INFEASIBLE with *out = NULL and info filled.
 */
int dq_build_tables(const dq_config* cfg, dq_tables** out, dq_table_info* info);
void dq_free_tables(dq_tables* tables);

/*
 * Encodes new tokens into records (Fig. 1; Alg. 1 and the rANS coder).
 *   kv:      bf16 [batch][tokens][kv_heads][head_dim] at element strides
 *            (stride_b, stride_t, stride_h); channels contiguous.  Token i of
 *            the input becomes cache token t0 + i.
 *   records: u8 [batch][kv_heads][t_cap][C]; writes tokens [t0, t0 + n_new).
 *   mean_q, mean_scale: keys only -- int8 [batch][kv_heads][t_cap/128][head_dim]
 *            and fp16 [batch][kv_heads][t_cap/128]: the per-window INT8
 *            channel mean of the rotated keys, which is removed before
 *            quantization (Sec. 4.2).  Both NULL for values (no mean removal);
 *            with them, t0 and n_new must be multiples of 128.
 *   status:  device u32, may be NULL; DQ_STATUS_RANGE / DQ_STATUS_OVERFLOW.
 * Every stream is rotated with the unnormalized Sylvester Hadamard matrix,
 * unless the tables were built with prerotated = 1 (then the input is coded
 * as it is).  The records are bit-identical to the reference definition of
 * the format.
 * Requires head_dim <= 256, 1 <= kv_heads <= 65535, 0 <= batch <= 65535,
 * t0 >= 0, n_new >= 0, t0 + n_new <= t_cap and non-negative strides; with the
 * mean buffers also t0, n_new and t_cap multiples of 128.  Returns DQ_OK
 * (nothing is launched when batch or n_new is 0), DQ_ERR_INVALID_ARG, or
 * DQ_ERR_HIP if a launch fails.
 */
int dq_encode_kv(const dq_tables* tables, const uint16_t* kv, int64_t stride_b,
                 int64_t stride_t, int64_t stride_h, int32_t batch,
                 int32_t kv_heads, int32_t t0, int32_t n_new, int32_t t_cap,
                 uint8_t* records, int8_t* mean_q, uint16_t* mean_scale,
                 uint32_t* status, void* stream);

/* Workspace bytes dq_decode_attention needs for these sizes. */
size_t dq_decode_workspace_bytes(int32_t batch, int32_t q_heads, int32_t kv_heads,
                                 int32_t t_cap, int32_t head_dim);

/*
 * One decode step of attention over the compressed cache (Sec. 4.5 decoding,
 * App. A): logits softmax_scale * q . k_hat over the first seq_lens[b] tokens,
 * output sum_t a_t v_hat_t, with query head i reading KV head
 * i / (q_heads / kv_heads).  q and out are in the basis the caller gives keys
 * and values in: with online rotation (prerotated = 0) that is the original
 * basis (the query is rotated and the output rotated back inside); with
 * prerotated keys the query must come in the keys' basis, and with
 * prerotated values the output stays in the values' basis (the caller's
 * output projection absorbs the rotation).  The raw tokens of a residual
 * window are taken in the same bases.
 *   q:        bf16 [batch][q_heads][head_dim]
 *   k_records, v_records: u8 [batch][kv_heads][t_cap][C_k or C_v]
 *   k_mean_q, k_mean_scale: as written by dq_encode_kv for the keys
 *   seq_lens: device int32 [batch], each in [0, t_cap]
 *   out:      fp32 [batch][q_heads][head_dim] (a sequence of length 0 gives 0)
 *   workspace: device memory of dq_decode_workspace_bytes(...) bytes
 *   status:   device u32, may be NULL; DQ_STATUS_CORRUPT for malformed records
 * Requires head_dim = 128 for both tables, record lengths C_k and C_v that
 * are multiples of 4 in [12, 64], t_cap a positive multiple of 128,
 * 1 <= batch <= 65535, 1 <= kv_heads <= 65535, q_heads a multiple of kv_heads
 * with q_heads / kv_heads <= 8.  Returns DQ_OK, DQ_ERR_INVALID_ARG (nothing
 * launched), DQ_ERR_WORKSPACE (workspace missing or too small) or DQ_ERR_HIP.
 */
int dq_decode_attention(const dq_tables* k_tables, const dq_tables* v_tables,
                        const uint16_t* q, int32_t batch, int32_t q_heads,
                        int32_t kv_heads, const uint8_t* k_records,
                        const int8_t* k_mean_q, const uint16_t* k_mean_scale,
                        const uint8_t* v_records, const int32_t* seq_lens,
                        int32_t t_cap, float softmax_scale, float* out,
                        void* workspace, size_t workspace_bytes,
                        uint32_t* status, void* stream);

/*
 * dq_decode_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops and
 * harnesses that forbid hipMalloc).  The split-K workspace lives in a static
 * device array of DQ_NO_ALLOC_SCRATCH_BYTES inside the library, one per
 * device, held until the process ends; its address is looked up on the first
 * call on each device (with that device current).  Arguments, layouts,
 * results and status bits are those of dq_decode_attention, and the same
 * kernels run.  No call allocates or frees memory.
 * Every call on a device shares that device's array, which keeps the last
 * call's contents: calls that overlap on one device (different streams, or
 * different host threads) race and give undefined results; serialize them.
 * The workspace this needs is 256 + 520 batch q_heads (chunks + 4) bytes,
 * chunks being the context split chosen from (batch, kv_heads, t_cap) and the
 * CU count (2 for 16 x 32768 tokens x 8 KV heads on 256 CUs: 1.6 MB).
 * Returns DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE when the sizes need more
 * than the array holds (dq_last_error says how much), or DQ_ERR_HIP.
 */
#define DQ_NO_ALLOC_SCRATCH_BYTES (8u << 20)
int dq_decode_attention_no_alloc(const dq_tables* k_tables, const dq_tables* v_tables,
                                 const uint16_t* q, int32_t batch, int32_t q_heads,
                                 int32_t kv_heads, const uint8_t* k_records,
                                 const int8_t* k_mean_q, const uint16_t* k_mean_scale,
                                 const uint8_t* v_records, const int32_t* seq_lens,
                                 int32_t t_cap, float softmax_scale, float* out,
                                 uint32_t* status, void* stream);

/*
 * The two halves of dq_decode_attention, for callers that merge partial
 * results themselves (e.g. context split over devices) or time them apart.
 * _partial writes one (max, sum, accumulator) triple per (sequence, query
 * head, context chunk) into the workspace (online-softmax state over the
 * chunk); _merge combines the chunks by log-sum-exp, undoes the value
 * rotation and writes `out`.  Arguments mean what they mean above; the chunk
 * size is chosen from (batch, kv_heads, t_cap) and the device's CU count and
 * recorded in the workspace, so both halves must be called with the same
 * sizes and workspace, on the same device and stream.
 */
int dq_decode_attention_partial(const dq_tables* k_tables, const dq_tables* v_tables,
                                const uint16_t* q, int32_t batch, int32_t q_heads,
                                int32_t kv_heads, const uint8_t* k_records,
                                const int8_t* k_mean_q, const uint16_t* k_mean_scale,
                                const uint8_t* v_records, const int32_t* seq_lens,
                                int32_t t_cap, float softmax_scale, void* workspace,
                                size_t workspace_bytes, uint32_t* status, void* stream);
int dq_decode_attention_merge(int32_t batch, int32_t q_heads, int32_t kv_heads,
                              const int32_t* seq_lens, int32_t t_cap, const void* workspace,
                              size_t workspace_bytes, float* out, void* stream);

/*
 * Residual window (Sec. 5.1 keeps the most recent tokens in BF16).  The raw
 * keys and values of a sequence's newest tokens live in a ring:
 *   res_k, res_v: bf16 [batch][kv_heads][r_cap][head_dim], 16-byte aligned,
 *            r_cap <= 256; residual token i of sequence b sits in slot
 *            (seq_lens[b] + i) mod r_cap, in the original basis (no
 *            rotation, no mean removal).
 *   seq_lens: device int32 [batch], the compressed tokens of each sequence;
 *   res_lens: device int32 [batch], its residual tokens (<= r_cap).
 * With r_cap a multiple of 128 and seq_lens[b] a multiple of 128, the oldest
 * 128 residual tokens are the contiguous slots [seq_lens[b] mod r_cap, + 128):
 * encode them with dq_encode_kv at t0 = seq_lens[b] (element strides
 * r_cap * head_dim between heads and head_dim between tokens), then call
 * dq_residual_commit(..., 128).
 *
 * dq_decode_attention_residual writes the residual window's softmax partial
 * into the workspace: call it after dq_decode_attention_partial and before
 * dq_decode_attention_merge, with the same sizes and workspace; the merge then
 * attends over the compressed tokens and the residual tokens together
 * (a sequence with neither gives 0).  head_dim is 128; q_heads / kv_heads <= 8;
 * q, res_k and res_v 16-byte aligned.
 * Returns DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE or DQ_ERR_HIP.
 */
int dq_decode_attention_residual(const uint16_t* q, int32_t batch, int32_t q_heads,
                                 int32_t kv_heads, const uint16_t* res_k,
                                 const uint16_t* res_v, const int32_t* seq_lens,
                                 const int32_t* res_lens, int32_t r_cap, int32_t t_cap,
                                 float softmax_scale, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * The residual window and the merge in one launch (Sec. 5.1, Alg. 2): after
 * dq_decode_attention_partial (or any other _partial call) with the same
 * sizes and workspace, writes `out` as dq_decode_attention_residual followed
 * by dq_decode_attention_merge would (equal up to fp32 rounding order), one
 * kernel instead of two.  The workspace is read, not written, so the
 * residual slots it holds for the two-call form are ignored.  Arguments as
 * for the two calls; q 16-byte aligned (as for dq_decode_attention_residual).
 * Returns DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE or DQ_ERR_HIP.
 */
int dq_decode_attention_merge_residual(const uint16_t* q, int32_t batch, int32_t q_heads,
                                       int32_t kv_heads, const uint16_t* res_k,
                                       const uint16_t* res_v, const int32_t* seq_lens,
                                       const int32_t* res_lens, int32_t r_cap, int32_t t_cap,
                                       float softmax_scale, const void* workspace,
                                       size_t workspace_bytes, float* out, void* stream);

/*
 * Appends one token per sequence to its ring: k_new, v_new bf16
 * [batch][kv_heads][head_dim] go to slot (seq_lens[b] + res_lens[b]) mod
 * r_cap, and res_lens[b] grows by one.  A full ring is left unchanged and
 * sets DQ_STATUS_WINDOW.  Returns DQ_OK, DQ_ERR_INVALID_ARG or DQ_ERR_HIP.
 */
int dq_residual_append(const uint16_t* k_new, const uint16_t* v_new, int32_t batch,
                       int32_t kv_heads, int32_t head_dim, uint16_t* res_k, uint16_t* res_v,
                       const int32_t* seq_lens, int32_t* res_lens, int32_t r_cap,
                       uint32_t* status, void* stream);

/*
 * The oldest n residual tokens of every sequence have been encoded:
 * seq_lens[b] += n, res_lens[b] -= n.  A sequence holding fewer than n is
 * left unchanged and sets DQ_STATUS_WINDOW.
 */
int dq_residual_commit(int32_t* seq_lens, int32_t* res_lens, int32_t batch, int32_t n,
                       uint32_t* status, void* stream);

/*
 * Paged layout, for serving engines that allocate the cache in pages.  The
 * records and key means of every sequence live in fixed-size pages of a pool:
 *   record pools:    u8 [num_pages][kv_heads][page_tokens][C]
 *   mean_q pool:     int8 [num_pages][kv_heads][page_tokens/128][head_dim]
 *   mean_scale pool: fp16 [num_pages][kv_heads][page_tokens/128]
 *   block_table:     device int32 [batch][max_pages]; logical page i of
 *                    sequence b (tokens [i page_tokens, (i+1) page_tokens)) is
 *                    pool page block_table[b * max_pages + i].
 * page_tokens is a power of two in [128, 2^20]; the logical capacity t_cap =
 * max_pages * page_tokens takes the place of t_cap above (workspace size,
 * the merge).  Otherwise the calls mean what their contiguous forms mean.  A
 * block-table entry outside [0, num_pages) sets DQ_STATUS_PAGE: the encoder
 * writes nothing through it, the attention reads page 0 in its place.
 */
int dq_encode_kv_paged(const dq_tables* tables, const uint16_t* kv, int64_t stride_b,
                       int64_t stride_t, int64_t stride_h, int32_t batch, int32_t kv_heads,
                       int32_t t0, int32_t n_new, const int32_t* block_table,
                       int32_t max_pages, int32_t page_tokens, int32_t num_pages,
                       uint8_t* record_pool, int8_t* mean_q_pool, uint16_t* mean_scale_pool,
                       uint32_t* status, void* stream);
int dq_decode_attention_paged_partial(const dq_tables* k_tables, const dq_tables* v_tables,
                                      const uint16_t* q, int32_t batch, int32_t q_heads,
                                      int32_t kv_heads, const uint8_t* k_pool,
                                      const int8_t* mean_q_pool, const uint16_t* mean_scale_pool,
                                      const uint8_t* v_pool, const int32_t* block_table,
                                      int32_t max_pages, int32_t page_tokens, int32_t num_pages,
                                      const int32_t* seq_lens, float softmax_scale,
                                      void* workspace, size_t workspace_bytes, uint32_t* status,
                                      void* stream);

/*
 * Per-token streams (Sec. 4.1, Sec. 4.5 "Decoding", Sec. 5.1): the paper's
 * default grouping, one stream of n = 128 kv_heads values per token spanning
 * every KV head (e.g. 1024 values for 8 heads, with 331 + 4 and 231 + 4 byte
 * records), instead of one stream per (token, KV head).  The stream takes the
 * heads in order, each head rotated on its own and, for keys, minus its own
 * window mean (the means are per head exactly as above); one (s, o) header
 * serves the whole token.  Tables are built with head_dim = n = 128 kv_heads.
 *
 * dq_token_record_stride: bytes of one token's record slot S, C rounded up to
 *   a multiple of 16 (the pad bytes are written as zeros); 0 for an invalid
 *   table.
 * Record buffer: u8 [batch][t_cap / 64][S / 8][64][8], 16-byte aligned: per
 *   64-token tile, the 8-byte chunks of the 64 records with the chunk index
 *   outermost (byte k of token t in tile t / 64 at ((k / 8) 64 + t % 64) 8 +
 *   k % 8), so that the 64 tokens' chunk k / 8 are 512 contiguous bytes.
 * dq_encode_kv_token: as dq_encode_kv with kv_heads in {1, 2, 4, 8} and
 *   head_dim 128; writes the record buffer above.
 * dq_decode_attention_token_partial: one decode step over those records
 *   (rANS-decoded once per token and consumed one KV head at a time), into the
 *   workspace of dq_decode_workspace_bytes; finish with
 *   dq_decode_attention_merge (and optionally add a residual window with
 *   dq_decode_attention_residual before it).  q_heads / kv_heads <= 8;
 *   k_mean_q / k_mean_scale as for dq_decode_attention.  Corrupt records set
 *   DQ_STATUS_CORRUPT.
 * Return DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE or DQ_ERR_HIP.
 */
int32_t dq_token_record_stride(const dq_tables* tables);
int dq_encode_kv_token(const dq_tables* tables, const uint16_t* kv, int64_t stride_b,
                       int64_t stride_t, int64_t stride_h, int32_t batch, int32_t kv_heads,
                       int32_t t0, int32_t n_new, int32_t t_cap, uint8_t* records,
                       int8_t* mean_q, uint16_t* mean_scale, uint32_t* status, void* stream);
int dq_decode_attention_token_partial(const dq_tables* k_tables, const dq_tables* v_tables,
                                      const uint16_t* q, int32_t batch, int32_t q_heads,
                                      int32_t kv_heads, const uint8_t* k_records,
                                      const int8_t* k_mean_q, const uint16_t* k_mean_scale,
                                      const uint8_t* v_records, const int32_t* seq_lens,
                                      int32_t t_cap, float softmax_scale, void* workspace,
                                      size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * Per-token records in pool pages (the paged layout above, Sec. 4.1's fixed
 * stride kept within a page): a pool page holds the records of page_tokens
 * tokens in the tile layout of the record buffer, so the record pool is
 * u8 [num_pages][page_tokens / 64][S / 8][64][8] and token t of sequence b is
 * row t mod page_tokens of pool page block_table[b * max_pages + t /
 * page_tokens].  Key-mean pools, the block table, page_tokens, the logical
 * capacity and DQ_STATUS_PAGE are as for dq_encode_kv_paged and
 * dq_decode_attention_paged_partial; otherwise the calls mean what
 * dq_encode_kv_token and dq_decode_attention_token_partial mean.
 */
int dq_encode_kv_token_paged(const dq_tables* tables, const uint16_t* kv, int64_t stride_b,
                             int64_t stride_t, int64_t stride_h, int32_t batch, int32_t kv_heads,
                             int32_t t0, int32_t n_new, const int32_t* block_table,
                             int32_t max_pages, int32_t page_tokens, int32_t num_pages,
                             uint8_t* record_pool, int8_t* mean_q_pool, uint16_t* mean_scale_pool,
                             uint32_t* status, void* stream);
int dq_decode_attention_token_paged_partial(const dq_tables* k_tables, const dq_tables* v_tables,
                                            const uint16_t* q, int32_t batch, int32_t q_heads,
                                            int32_t kv_heads, const uint8_t* k_pool,
                                            const int8_t* mean_q_pool, const uint16_t* mean_scale_pool,
                                            const uint8_t* v_pool, const int32_t* block_table,
                                            int32_t max_pages, int32_t page_tokens, int32_t num_pages,
                                            const int32_t* seq_lens, float softmax_scale,
                                            void* workspace, size_t workspace_bytes, uint32_t* status,
                                            void* stream);

/*
 * Comparator: fixed-width coding at matched storage (App. B).  The same
 * preprocessing as the D-Quant encoder (rotation, key window means, min-max
 * grid, least-squares refit, fp16 s and o), symbols by nearest-level rounding,
 * b = floor(8 (record_bytes - 4) / head_dim) bits each (M = 2^b levels),
 * packed least-significant bit first after the 4-byte header of a record of
 * the same size.  With 36-byte records and head_dim 128 that is 128 two-bit
 * codes sharing one fp16 scale and one fp16 offset: 2.25 bits per value, the
 * 2-bit example of Sec. 3.
 *
 * dq_fixed_bits: b for (head_dim, record_bytes), 0 if no whole bit fits or
 *   more than 8 would.
 * dq_encode_kv_fixed: as dq_encode_kv without tables; head_dim 64, 128 or 256.
 * dq_decode_attention_fixed_partial: one decode step over 36-byte fixed-width
 *   records (head_dim 128, b = 2), same layouts, workspace and merge as
 *   dq_decode_attention_partial; q_heads / kv_heads <= 4.
 * Return DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE or DQ_ERR_HIP.
 */
int32_t dq_fixed_bits(int32_t head_dim, int32_t record_bytes);
int dq_encode_kv_fixed(int32_t head_dim, int32_t record_bytes, const uint16_t* kv, int64_t stride_b,
                       int64_t stride_t, int64_t stride_h, int32_t batch, int32_t kv_heads, int32_t t0,
                       int32_t n_new, int32_t t_cap, uint8_t* records, int8_t* mean_q,
                       uint16_t* mean_scale, uint32_t* status, void* stream);
int dq_decode_attention_fixed_partial(const uint16_t* q, int32_t batch, int32_t q_heads, int32_t kv_heads,
                                      const uint8_t* k_records, const int8_t* k_mean_q,
                                      const uint16_t* k_mean_scale, const uint8_t* v_records,
                                      const int32_t* seq_lens, int32_t t_cap, float softmax_scale,
                                      void* workspace, size_t workspace_bytes, uint32_t* status,
                                      void* stream);

/*
 * Comparator: the same decode step over an uncompressed BF16 cache.
 *   k, v: bf16 [batch][kv_heads][t_cap][head_dim], 16-byte aligned, original
 *         basis; the first seq_lens[b] tokens of sequence b are attended.
 * Writes split-K partials into the workspace (same size rule as above);
 * finish with dq_decode_attention_merge, with the same sizes and workspace.
 * head_dim is 128; t_cap a positive multiple of 128; q_heads / kv_heads <= 8.
 * Returns DQ_OK, DQ_ERR_INVALID_ARG, DQ_ERR_WORKSPACE or DQ_ERR_HIP.
 */
int dq_bf16_decode_attention_partial(const uint16_t* q, int32_t batch, int32_t q_heads,
                                     int32_t kv_heads, const uint16_t* k, const uint16_t* v,
                                     const int32_t* seq_lens, int32_t t_cap,
                                     float softmax_scale, void* workspace,
                                     size_t workspace_bytes, void* stream);

/*
 * rANS-decodes records back to symbols (Alg. 2), for parity checks.
 *   records: u8 [n_streams][C]; sym: u8 [n_streams][head_dim];
 *   header:  u16 [n_streams][2] = (scale, offset) fp16 bits; may be NULL;
 *   status:  DQ_STATUS_CORRUPT if a record is malformed; may be NULL.
 */
int dq_decode_symbols(const dq_tables* tables, const uint8_t* records,
                      int64_t n_streams, uint8_t* sym, uint16_t* header,
                      uint32_t* status, void* stream);

/* Static description of a return code. */
const char* dq_strerror(int code);

/* The HIP call that last failed in this thread with DQ_ERR_HIP, and its HIP
 * error name and text ("" if none).  Valid until the next failing call. */
const char* dq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DQ_H */
