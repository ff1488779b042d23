// Internal definitions shared by the host library and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dq.h"

namespace dq {

constexpr uint32_t kRansL = 1u << 21;       // rANS lower bound; state in [L, 256 L)
constexpr int kLambdaSteps = 512;           // lambda grid points per octave
constexpr int kPayloadOffset = 8;           // fp16 scale, fp16 offset, u32 state
constexpr int kBisectSteps = 12;            // T of Alg. 1
constexpr int kBracketUnits = 40 * kLambdaSteps;  // hi - lo = 40 octaves

// Split-K attention workspace: a 256-byte header (chunk size, chunk count NC,
// residual slots written), then fp32 acc [B][Hq][NC + kResSlots][d], m and l
// [B][Hq][NC + kResSlots], sized for chunks of at least kMinChunk tokens
// (per-token streams; the per-head and BF16 kernels take chunks of at least
// kMinChunkHead).  Slots NC .. NC + kResSlots - 1 of each (sequence, query
// head) hold the residual window's partials, one per workgroup of its split.
constexpr int kWsHeader = 256;
constexpr int kMinChunk = 128;
constexpr int kMinChunkHead = 256;
constexpr int kResSlots = 4;
inline int64_t max_chunks(int t_cap) { return (t_cap + kMinChunk - 1) / kMinChunk; }
inline int64_t ws_slots(int B, int Hq, int t_cap) { return (int64_t)B * Hq * (max_chunks(t_cap) + kResSlots); }
int cu_count();   // CUs of the current device

// Where the records and key means of (sequence b, KV head h, token t) live.
//   contiguous (bt == NULL): records [B][H][t_cap][C], means [B][H][t_cap/128][.]
//   paged: pools [num_pages][H][page][C] and [num_pages][H][page/128][.]; the
//          logical page i of sequence b is the physical page bt[b * max_pages + i],
//          page = 2^page_shift >= 128 tokens, t_cap = max_pages * page.
// A block-table entry outside [0, num_pages) reads page 0 and raises *bad.
struct Pages {
    const int32_t* bt;
    int32_t max_pages;
    int32_t page_shift;
    int32_t num_pages;
};

__device__ __forceinline__ int32_t physical_page(const Pages& pg, int b, int t, bool& bad) {
    int32_t p = pg.bt[(int64_t)b * pg.max_pages + (t >> pg.page_shift)];
    if (p < 0 || p >= pg.num_pages) {
        bad = true;
        p = 0;
    }
    return p;
}

// Record row (index in units of one record) of token t; rows of the tokens of
// an aligned 64-token tile are consecutive.
__device__ __forceinline__ int64_t record_row(const Pages& pg, int H, int t_cap, int b, int h, int t, bool& bad) {
    if (!pg.bt) return ((int64_t)b * H + h) * t_cap + t;
    const int64_t p = physical_page(pg, b, t, bad);
    return ((p * H + h) << pg.page_shift) + (t & ((1 << pg.page_shift) - 1));
}

// Row of token t of sequence b in a per-token record buffer, whose rows hold
// the records of all heads of one token: b t_cap + t, or row t mod page of
// pool page p (rows p page .. p page + page - 1).  A page holds whole
// 64-token tiles.
__device__ __forceinline__ int64_t token_row(const Pages& pg, int t_cap, int b, int t, bool& bad) {
    if (!pg.bt) return (int64_t)b * t_cap + t;
    const int64_t p = physical_page(pg, b, t, bad);
    return (p << pg.page_shift) + (t & ((1 << pg.page_shift) - 1));
}

// Index of the 128-token mean window w of (b, h).
__device__ __forceinline__ int64_t window_index(const Pages& pg, int H, int t_cap, int b, int h, int w, bool& bad) {
    if (!pg.bt) return ((int64_t)b * H + h) * (t_cap / DQ_MEAN_WINDOW) + w;
    const int t = w * DQ_MEAN_WINDOW;
    const int64_t p = physical_page(pg, b, t, bad);
    const int wpp = 1 << (pg.page_shift - 7);
    return (p * H + h) * wpp + ((t & ((1 << pg.page_shift) - 1)) >> 7);
}

// Device-resident tables, one allocation.
//   lut[z], z in [0, 2^p):  bias (z - c_m) in bits 0..11, f_m in bits 12..23,
//                           m in bits 24..29.
//   lut64[z]: x = 8 f_m | m << 24 (a 24-bit multiply reads 8 f_m), y = 8 (z - c_m).
struct DevTables {
    const uint32_t* lut;
    const uint2* lut64;
    const int32_t* freq;
    const int32_t* cum;
    const int32_t* cost;   // Q16
    const float* lam;      // [512]
};

// Everything a kernel needs about one coding configuration (by value).
struct TabArgs {
    DevTables t;
    int32_t n;          // values per stream
    int32_t M;          // levels
    int32_t p;          // precision bits
    int32_t C;          // record bytes
    int32_t cheapest;   // lowest-index minimum-cost symbol
    int32_t rmin;       // minimum cost (Q16)
    int64_t budget;     // Q16 budget
};

}  // namespace dq

struct dq_tables {
    dq_config cfg;
    dq_table_info info;
    int32_t freq[DQ_MAX_LEVELS];
    int32_t cum[DQ_MAX_LEVELS];
    int32_t cost[DQ_MAX_LEVELS];
    int device;
    void* dev_block;
    dq::DevTables dev;
};

namespace dq {

inline TabArgs tab_args(const dq_tables* t) {
    TabArgs a;
    a.t = t->dev;
    a.n = t->cfg.head_dim;
    a.M = t->cfg.levels;
    a.p = t->cfg.precision_bits;
    a.C = t->cfg.record_bytes;
    a.cheapest = t->info.cheapest;
    int32_t rmin = t->cost[0];
    for (int m = 1; m < t->cfg.levels; ++m) rmin = t->cost[m] < rmin ? t->cost[m] : rmin;
    a.rmin = rmin;
    a.budget = t->info.budget_q16;
    return a;
}

// Records the failing HIP call for dq_last_error(); returns DQ_ERR_HIP.
int hip_fail(const char* where, hipError_t err);

// DQ_OK if err is hipSuccess, else records it and returns DQ_ERR_HIP.
inline int hip_check(const char* where, hipError_t err) {
    return err == hipSuccess ? DQ_OK : hip_fail(where, err);
}

// Launchers implemented in the .hip files.  Return DQ_OK or DQ_ERR_HIP.
// token_stride > 0: one stream per token over the H heads (head_dim 128, the
// table's n = 128 H), records [B][t_cap][token_stride]; 0: per (token, head).
int launch_encode(const dq_tables* tab, const Pages& pg, const uint16_t* kv, int64_t sb, int64_t st,
                  int64_t sh, int32_t B, int32_t H, int32_t t0, int32_t n_new,
                  int32_t t_cap, uint8_t* records, int8_t* mean_q,
                  uint16_t* mean_scale, uint32_t* status, hipStream_t stream, int token_stride = 0);

int launch_decode_symbols(const dq_tables* tab, const uint8_t* records, int64_t n_streams,
                          uint8_t* sym, uint16_t* header, uint32_t* status,
                          hipStream_t stream);

size_t attention_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap, int32_t d);

// ws_slots_used: (max, sum, accumulator) slots the workspace holds, which
// places the max and sum arrays after the accumulators; 0 = the size
// attention_workspace_bytes allows for (chunks of kMinChunk tokens).
int launch_attention_partial(const dq_tables* tk, const dq_tables* tv, const Pages& pg, const uint16_t* q,
                             int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* krec,
                             const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                             const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                             uint32_t* status, hipStream_t stream, int64_t ws_slots_used = 0);

// Slots the chunk plan of these sizes uses on the current device:
// B Hq (chunks + kResSlots), the last ones per query head for the residual
// window.
int64_t attention_plan_slots(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap);

// Device address of the current device's copy of the library's static
// scratch array (DQ_NO_ALLOC_SCRATCH_BYTES), looked up once per device.
int no_alloc_scratch(void** out);
constexpr int kMaxDevices = 64;

// Per-token streams over Hkv heads (table n = 128 Hkv, G = Hq / Hkv <= 8),
// records [B][t_cap][stride] in 64-token tiles, or token rows of pool pages
// through pg; same workspace as launch_attention_partial.
int launch_attention_token_partial(const dq_tables* tk, const dq_tables* tv, const Pages& pg, const uint16_t* q,
                                   int32_t B,
                                   int32_t Hq, int32_t Hkv, const uint8_t* krec, int32_t k_stride,
                                   const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                                   int32_t v_stride, const int32_t* seq_lens, int32_t t_cap, float scale,
                                   void* ws, uint32_t* status, hipStream_t stream);
int32_t token_chunk(int32_t B, int32_t t_cap);

// Fixed-width comparator (App. B): 36-byte records of 128 2-bit levels
// ([fp16 s][fp16 o][32 payload bytes]), head_dim 128, G <= 4; same workspace.
constexpr int kFixedRecordBytes = 36;
int launch_attention_fixed_partial(const Pages& pg, const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                   const uint8_t* krec, const int8_t* kmq, const uint16_t* kms,
                                   const uint8_t* vrec, const int32_t* seq_lens, int32_t t_cap, float scale,
                                   void* ws, uint32_t* status, hipStream_t stream);
// Fixed-width encoder: same preprocessing, nearest-level rounding, b-bit
// symbols packed after the 4-byte header of a C-byte record.
int launch_encode_fixed(int32_t n, int32_t record_bytes, const Pages& pg, const uint16_t* kv, int64_t sb,
                        int64_t st, int64_t sh, int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                        uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status,
                        hipStream_t stream);

int launch_attention_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                              const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                              const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                              void* ws, hipStream_t stream);
int launch_attention_merge_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                    const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                                    const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                                    void* ws, float* out, hipStream_t stream);
int launch_residual_append(const uint16_t* k_new, const uint16_t* v_new, int32_t B, int32_t Hkv,
                           uint16_t* res_k, uint16_t* res_v, const int32_t* seq_lens, int32_t* res_lens,
                           int32_t r_cap, uint32_t* status, hipStream_t stream);
int launch_residual_commit(int32_t* seq_lens, int32_t* res_lens, int32_t B, int32_t n, uint32_t* status,
                           hipStream_t stream);
int launch_bf16_partial(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, const uint16_t* k,
                        const uint16_t* v, const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                        hipStream_t stream);
int launch_attention_merge(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* seq_lens,
                           int32_t t_cap, const void* ws, float* out, hipStream_t stream,
                           int64_t ws_slots_used = 0);

}  // namespace dq
