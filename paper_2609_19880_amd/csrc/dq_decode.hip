// Decode side: rANS decoding of the fixed-size records (Alg. 2) and decode
// attention over them (Sec. 4.5 "Decoding", App. A Eq. fold-key/fold-value).
//
// decode_attention is split-K over context chunks:
//  * attn_partial: one workgroup per (chunk, KV head, sequence), up to 12
//    wavefronts.  The workgroup stages the rANS tables in LDS and rotates the
//    G query heads that share the KV head (one FWHT in LDS).  Each wavefront
//    then takes 64-token tiles, one token per lane: the lane stages its key
//    and value payloads in LDS and runs the two rANS chains interleaved.  Key
//    levels feed the q . k products on the matrix cores as they are decoded
//    (Eq. fold-key); value levels wait in registers until the tile's softmax
//    weights are known, then meet them on the matrix cores (Eq. fold-value).
//    Online softmax state stays per wavefront; the wavefronts are merged in
//    LDS at the end.
//  * attn_merge: log-sum-exp merge of the chunk partials per (sequence, query
//    head), then the inverse rotation of the value basis and the 1/d scale.
#include <math.h>

#include <algorithm>
#include <mutex>

#include "dq_attn.h"

namespace dq {
namespace {

constexpr int kD = 128;          // head_dim of the attention kernels
constexpr int kTile = 64;        // tokens per wavefront tile (one per lane)
constexpr int kMaxWaves = 16;    // wavefronts per workgroup (LDS permitting)
constexpr int kVSlice = 64;      // value channels per PV pass
constexpr int kVRowT = 80;       // bytes per token row of the value tile (64 channels + pad)
constexpr int kMaxRecDwords = 16;
constexpr int kMaxLds = 160 * 1024;
constexpr int kMaxChunk = 16384;  // bounds the per-window q . mu table in LDS

// ---------------------------------------------------------------- symbols

__global__ void decode_symbols_kernel(TabArgs ta, const uint8_t* __restrict__ rec, int64_t S,
                                      uint8_t* __restrict__ sym, uint16_t* __restrict__ hdr,
                                      uint32_t* status) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S) return;
    const int C = ta.C;
    const uint8_t* r = rec + s * C;
    uint32_t x = (uint32_t)r[4] | ((uint32_t)r[5] << 8) | ((uint32_t)r[6] << 16) |
                 ((uint32_t)r[7] << 24);
    int ptr = kPayloadOffset;
    const uint32_t mask = (1u << ta.p) - 1u;
    uint8_t* out = sym + s * ta.n;
    for (int j = 0; j < ta.n; ++j) {
        const uint32_t e = ta.t.lut[x & mask];
        x = ((e >> 12) & 0xFFFu) * (x >> ta.p) + (e & 0xFFFu);
        while (x < kRansL && ptr < C) {
            x = (x << 8) | r[ptr];
            ++ptr;
        }
        out[j] = (uint8_t)(e >> 24);
    }
    if (hdr) {
        hdr[2 * s] = (uint16_t)(r[0] | (r[1] << 8));
        hdr[2 * s + 1] = (uint16_t)(r[2] | (r[3] << 8));
    }
    if ((x != kRansL) && status) atomicOr(status, DQ_STATUS_CORRUPT);
}

// -------------------------------------------------------------- attention
//
// Work split.  One workgroup per (context chunk, KV head, sequence); each
// wavefront takes 64-token tiles, one token per lane, and decodes that
// token's key stream then its value stream (Alg. 2), 128 steps each.
//
// Decode step.  The state is kept as X = 8 x (its low three bits are never
// read), which with 8-byte table entries (f_m | m << 24, z - c_m) in LDS
// makes the table address one mask of X and the state update
// x' = f (x >> p) + (z - c) one 24-bit multiply-add.  Renormalization bytes
// are staged per lane as overlapping big-endian byte pairs
// P[k] = (b_k << 8) | b_{k+1}: one aligned 16-bit LDS read yields the next
// 16 bits wherever the lane's byte pointer stands.  Since x' >= 2^9 for
// p <= 12, the number of bytes Alg. 2 reads (0, 1 or 2) is n = sh / 8 with
// sh = (clz(x') - 3) & 24, and with s = 29 - sh (13, 21 or 29)
//     X = alignbit(x', P[ptr] << 16, s) = (x' << (3 + sh)) | (P[ptr] << 16 >> s),
// whose first sh bits of the pair land at bit 3 (the low three bits are
// left-overs of the pair, never read).  The byte pointer advances by n
// positions of 128 bytes, 464 - 16 s bytes: the register holds the pointer
// less 464 j at step j of a 16-step window, so that it moves by -16 s and
// each read carries its 464 j as the instruction's offset.
//
// Contractions (Eq. fold-key / fold-value) run on the matrix cores.  Decoded
// levels are bytes and enter as they are; the rotated query and the softmax
// weights (with the value scale folded in) enter as three signed 8-bit digits
// of a 22-bit fixed-point value, accumulated exactly in int32 and recombined
// in fp32.
//   q . k:  v_mfma_i32_4x4x4_16b_i8 (16 blocks of 4x4x4; lane l is column
//           l % 4 of block l / 4), block = 4 tokens, K = 4 channels.  A = the
//           query digits of head l % 4, B = the 4 levels the lane just
//           decoded, D = the lane's own token's dot products for 4 heads.
//   P . v:  v_mfma_i32_16x16x32_i8, rows = (query-head slot, digit), K = 32
//           tokens, columns = 16 channels.  Each lane writes its token's
//           levels and weight digits to token-major LDS rows as they are, and
//           ds_read_b64_tr_b8 hands every lane the 8 tokens of one row or
//           column the product wants; D = one slot's three digit sums (and a
//           zero row) of channel l % 16.

struct AttnLayout {
    int nw;             // wavefronts per workgroup
    int lut_k, lut_v;   // 8-byte tables (the same offset when K and V share one)
    int qlimb;          // [32 channel groups][GP heads] x 16 B (three digit words)
    int qscale, qsum;   // float [GP]
    int qmu;            // float [windows][GP]
    int waves;          // first wavefront region
    int wave_stride;
    int pk, pv;             // key / value byte-pair arrays: [position][64 lanes] x 2 B
    int vtile;              // [64 tokens][kVRowT] level bytes of a 64-channel slice, over the pair arrays
    int plimb;              // [HG][64 tokens][16] weight digits: byte 4 slot + digit (digit 3: zero)
    int total;
};

__host__ inline int align16(int v) { return (v + 15) & ~15; }

constexpr int kPairRow = 2 * kTile;     // bytes per payload position: one pair per lane
constexpr int kPairSlack = 4096;         // LDS above the last array that a corrupt stream may read
constexpr int kClampGroups = 4;          // pointers are clamped every 4 x 4 decode steps
constexpr int kWindow = 4 * kClampGroups;            // decode steps per pointer window
constexpr int kPairStep = 29 * kPairRow / 8;         // 464: read offset per step of a window

struct AttnArgs {
    TabArgs tk, tv;
    const uint16_t* q;
    int Hq, Hkv, G, t_cap, chunk, nchunks;
    const uint8_t* krec;
    const int8_t* kmq;
    const uint16_t* kms;
    const uint8_t* vrec;
    const int32_t* seq_lens;
    float scale_log2;            // softmax_scale * log2(e) / d
    int32_t* ws_hdr;             // [0] chunk, [1] chunk count NC, [2] residual slots written,
                                 // [3] 1 if the merge rotates the output back (values rotated online)
    int rot_q, rot_out;          // keys / values rotated online (tables not prerotated)
    float* ws_m;                 // [B][Hq][NC + kResSlots]   (slots NC..: the residual window)
    float* ws_l;                 // [B][Hq][NC + kResSlots]
    float* ws_acc;               // [B][Hq][NC + kResSlots][d]
    uint32_t* status;
    int shared_lut;
    Pages pg;                    // records and key means: contiguous or paged
    AttnLayout L;
};


// One step of Alg. 2 on the state kept as X = 8 x (+ up to 7 in the low bits,
// which nothing reads), in two halves so that the key and value chains of a
// lane overlap: the reads of one chain are in flight while the other's
// arithmetic runs.
//   table address = X & (2^p - 1) << 3          (8-byte entries at lut_off)
//   y = f (X >> (p + 3)) + (z - c) = x'          (one 24-bit multiply-add)
//   s = ((clz(y) - 3) & 24) ^ 29 = 29 - 8 n      (n = 0, 1 or 2 bytes to read)
//   X = alignbit(y, pair << 16, s),  Q -= 16 s   (J: step in the 16-step window,
//                                                  a constant once unrolled)
//
// dissue requests the pair (straight into the high half of r with
// ds_read_u16_d16_hi, which the compiler does not emit; the low half is never
// read) and the table word.  The compiler does not see these loads, so
// nothing may read r or e until dwait<N> has run on them: it waits until at
// most N LDS or scalar-memory operations are outstanding.  LDS returns in
// order, so N = the number of LDS reads issued after e in program order is
// enough (operations the compiler adds in between only make the wait
// stricter).  dfinish then completes the step and returns the table word
// (level in its top byte).
template <uint32_t LUT_OFF>
__device__ __forceinline__ void dissue(uint32_t X, uint32_t Q, uint32_t mask8, int J, uint32_t& r, uint64_t& e) {
    asm volatile("ds_read_u16_d16_hi %0, %2 offset:%4\n\t"
                 "ds_read_b64 %1, %3 offset:%5"
                 : "=&v"(r), "=&v"(e)
                 : "v"(Q), "v"(X & mask8), "i"(kPairStep * J), "i"(LUT_OFF));
}

template <int N>
__device__ __forceinline__ void dwait(uint32_t& r, uint64_t& e) {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(r), "+v"(e) : "i"(N));
}

// The query digits of one group (16 bytes at LDS address a + off, off a
// constant once unrolled), requested under the same rule: pending until a
// dwaitq that follows it has run.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void qissue(uint32_t a, int off, v4u& q) {
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=&v"(q) : "v"(a), "i"(off));
}

template <int N, int HG>
__device__ __forceinline__ void dwaitq(uint32_t& r, uint64_t& e, v4u (&q)[HG]) {
    if constexpr (HG == 1)
        asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(r), "+v"(e), "+v"(q[0]) : "i"(N));
    else
        asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(r), "+v"(e), "+v"(q[0]), "+v"(q[1]) : "i"(N));
}

// The query digits alone (a single chain whose next reads stay in flight).
template <int N>
__device__ __forceinline__ void dwaitq1(v4u& q) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(q) : "i"(N));
}

__device__ __forceinline__ uint32_t dfinish(uint32_t& X, uint32_t& Q, int p3, uint32_t r, uint64_t e) {
    const uint32_t ex = (uint32_t)e, ey = (uint32_t)(e >> 32);
    const uint32_t y = __umul24(ex, X >> p3) + ey;
    const uint32_t s = (((uint32_t)__builtin_clz(y) - 3u) & 24u) ^ 29u;
    X = __builtin_amdgcn_alignbit(y, r, s);
    asm("v_mad_i32_i24 %0, %1, -16, %2" : "=v"(Q) : "v"(s), "v"(Q));
    return ex;
}

// Copies a decode table into LDS: the device table holds 8 f | m << 24 and
// 8 (z - c), the decode step takes f | m << 24 and z - c.  Entries i0 + u nthr
// (u < 8) are requested by stage_load and stored by stage_store, so that the
// eight latencies overlap (and overlap whatever runs in between);
// stage_table copies entries i0 + 8 nthr on, eight per thread at a time.
__device__ __forceinline__ void stage_load(uint2 (&e)[8], const uint2* __restrict__ src, int n, int i0, int nthr) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
        if (i0 + u * nthr < n) e[u] = src[i0 + u * nthr];
}

__device__ __forceinline__ void stage_store(uint2* dst, const uint2 (&e)[8], int n, int i0, int nthr) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
        if (i0 + u * nthr < n)
            dst[i0 + u * nthr] = uint2{(e[u].x & 0xFF000000u) | ((e[u].x & 0x00FFFFFFu) >> 3), e[u].y >> 3};
}

__device__ __forceinline__ void stage_table(uint2* dst, const uint2* __restrict__ src, int n, int tid, int nthr) {
    for (int i0 = tid + 8 * nthr; i0 < n; i0 += 8 * nthr) {
        uint2 e[8];
        stage_load(e, src, n, i0, nthr);
        stage_store(dst, e, n, i0, nthr);
    }
}

// Record dwords of the lane's token (C % 4 == 0, C <= 64).
__device__ __forceinline__ void load_record(uint32_t (&r)[kMaxRecDwords], const uint8_t* recs,
                                            int64_t tok, int CW) {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(recs + tok * (CW * 4));
#pragma unroll
    for (int k = 0; k < kMaxRecDwords; ++k)
        if (k < CW) r[k] = src[k];
}

// Payload bytes of a record -> the lane's column of a byte-pair array: the
// big-endian pair (b_k << 8) | b_{k+1} of position k goes to dst + k * 128.
// A lane's pairs stay in one LDS bank whatever position it has reached.
__device__ __forceinline__ void build_pairs(const uint32_t (&r)[kMaxRecDwords], int CW, uint8_t* dst) {
#pragma unroll
    for (int k = 2; k < kMaxRecDwords; ++k) {
        if (k < CW) {
            const uint32_t w = r[k];
            const uint32_t wn = (k + 1 < CW) ? r[(k + 1) & (kMaxRecDwords - 1)] : 0u;
            const uint32_t d0 = __builtin_amdgcn_perm(w, w, 0x01020001u);
            const uint32_t d1 = __builtin_amdgcn_perm(wn, w, 0x03040203u);
            uint8_t* p = dst + 4 * (k - 2) * kPairRow;
            *reinterpret_cast<uint16_t*>(p) = (uint16_t)d0;
            *reinterpret_cast<uint16_t*>(p + kPairRow) = (uint16_t)(d0 >> 16);
            *reinterpret_cast<uint16_t*>(p + 2 * kPairRow) = (uint16_t)d1;
            *reinterpret_cast<uint16_t*>(p + 3 * kPairRow) = (uint16_t)(d1 >> 16);
        }
    }
}

// Wavefronts per workgroup (LDS permitting).  Up to 4 query heads per KV
// head: 16 (4 per SIMD, at most 128 VGPRs) for records of up to 36 bytes, 12
// for longer or run-time-length records, whose prefetched record words need
// more registers.  Up to 8 query heads: 12 (at most 168 VGPRs), without the
// record prefetch, whose registers the larger accumulators need; 8 for
// run-time record lengths.  When LDS holds no more than 8 wavefronts anyway
// (two 4096-entry tables), the 8-wavefront instantiation (256 VGPRs) keeps
// the prefetch.
// RWP packs the compile-time record lengths in dwords, keys << 8 | values
// (0: run-time lengths).
__host__ __device__ constexpr int rw_pair(int rwk, int rwv) { return (rwk << 8) | rwv; }
__host__ __device__ constexpr int max_waves(int HG, int RWP) {
    return HG == 1 ? ((RWP == rw_pair(8, 8) || RWP == rw_pair(9, 9)) ? kMaxWaves : 12) : (RWP ? 12 : 8);
}

constexpr uint32_t kLutVOffset = 8u << 12;   // value table when it differs from the key table

// RWP: compile-time key and value record lengths (rw_pair), 0 for run-time
// lengths.
// Fixed-width comparator records (App. B): [fp16 s][fp16 o] then 2-bit levels,
// symbol j in bits 2 (j mod 4) of payload byte j / 4.  The four levels of
// payload byte x, one per byte: x | (x >> 4) << 16 puts the two nibbles in
// the two halves, | << 6 brings bits 2-3 of each half up to its second byte.
__device__ __forceinline__ uint32_t spread2(uint32_t x) {
    uint32_t t, u;
    asm("v_lshl_or_b32 %0, %1, 16, %2" : "=v"(t) : "v"(x >> 4), "v"(x));
    asm("v_lshl_or_b32 %0, %1, 6, %1" : "=v"(u) : "v"(t));
    return u & 0x03030303u;
}

// FIXED: the fixed-width comparator at matched storage; levels come straight
// from the record words (no tables, no byte pairs, no rANS state).
// WMAX: the wavefront bound of the instantiation (max_waves, or 8).
// SPLIT: one tile per pair of wavefronts, keys and values decoded by
// different wavefronts (chunks of at most nw / 2 tiles: small batches).
template <int HG, uint32_t LUTV, int RWP, bool FIXED, int WMAX, bool SPLIT = false>
__global__ __launch_bounds__(WMAX * kWave) void attn_partial_kernel(AttnArgs a) {
    constexpr int RWK = RWP >> 8, RWV = RWP & 0xFF;
    constexpr int GP = 4 * HG;
    extern __shared__ __align__(16) uint8_t smem[];
    const AttnLayout& L = a.L;
    const int G = a.G;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int nthr = L.nw * kWave;
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    if ((c | h | b) == 0 && tid == 0) {
        a.ws_hdr[0] = a.chunk;
        a.ws_hdr[1] = a.nchunks;
        a.ws_hdr[2] = 0;          // set by the residual kernel when it runs
        a.ws_hdr[3] = a.rot_out;
    }
    // ---- the prologue's loads, all in flight together: the tables and the
    //      query heads (neither depends on the sequence's length), then the
    //      first tile's records and key means
    const int hq0 = h * G;
    // the tables go through the wavefronts that do not rotate a query head
    // when those can hold every entry in registers (8 per thread), else
    // through all of them
    const int Pk = 1 << a.tk.p, Pv = LUTV != 0 ? 1 << a.tv.p : 0;
    const int tw0 = (L.nw - G) * kWave * 8 >= max(Pk, Pv) ? G : 0;
    const int ttid = tid - tw0 * kWave, tthr = nthr - tw0 * kWave;
    uint2 lut_e[8], lutv_e[8];
    if (!FIXED && wave >= tw0) {
        stage_load(lut_e, a.tk.t.lut64, Pk, ttid, tthr);
        if (LUTV != 0) stage_load(lutv_e, a.tv.t.lut64, Pv, ttid, tthr);
    }
    // wavefront g < G rotates query head g (channels l and l + 64 in lane l)
    uint16_t qb0 = 0, qb1 = 0;
    if (wave < G) {
        const uint16_t* qh = a.q + ((int64_t)b * a.Hq + hq0 + wave) * kD;
        qb0 = qh[lane];
        qb1 = qh[lane + 64];
    }
    // records of the wavefront's first tile and key means of the first
    // window(s) of the q . mu table below.  In a contiguous cache every row
    // below t_cap exists, so they are requested before the sequence's length
    // is known (rows past it are loaded and not used); through a block table
    // only rows below the length may be looked up, so they wait for it.
    //   records: each later tile's records are requested once the tile before
    //     has its softmax weights, and arrive while its value products are
    //     formed (up to 4 query heads per KV head; with 8 the registers go to
    //     accumulators unless the workgroup has at most 8 wavefronts); a
    //     wavefront that turns out to have no tile may load one it does not
    //     use
    //   key means: half a wavefront per window, two windows per pass, lane l
    //     of wavefront nw - 1 - mw taking channels 4 (l % 32) .. + 3 of window
    //     2 (mw + pass nw) + l / 32 (the last wavefronts: the first ones form
    //     the query digits meanwhile)
    const int start = c * a.chunk;
    const bool paged = a.pg.bt != nullptr;
    const int Ck = RWK ? 4 * RWK : a.tk.C, Cv = RWV ? 4 * RWV : a.tv.C, CWk = Ck / 4, CWv = Cv / 4;
    constexpr bool kPrefetch = HG == 1 || WMAX <= 8;
    uint32_t rk[kMaxRecDwords], rv[kMaxRecDwords];
    const int nwin_total = a.t_cap / DQ_MEAN_WINDOW;
    const int w0 = start / DQ_MEAN_WINDOW;
    const int nwin = (a.chunk + DQ_MEAN_WINDOW - 1) / DQ_MEAN_WINDOW + 1;
    const int mwave = L.nw - 1 - wave;
    const int mwin = 2 * mwave + (lane >> 5);            // this lane's first window
    uint32_t mv0 = 0;
    uint16_t ms0 = 0;
    bool bad_page = false;
    // the wavefront's first tile (SPLIT: its pair's tile, keys in the even
    // wavefront with the value header, values in the odd one)
    const int ptile = SPLIT ? wave >> 1 : wave;
    const bool load_k = !SPLIT || !(wave & 1), load_v = !SPLIT || (wave & 1);
    if (!paged) {
        if (kPrefetch && ptile * kTile < a.chunk) {
            const int64_t tok = record_row(a.pg, a.Hkv, a.t_cap, b, h, min(start + ptile * kTile, a.t_cap - kTile),
                                           bad_page) + lane;
            if (load_k) load_record(rk, a.krec, tok, CWk);
            if (load_v) load_record(rv, a.vrec, tok, CWv);
            else rv[0] = *reinterpret_cast<const uint32_t*>(a.vrec + tok * (CWv * 4));
        }
        if (mwin < nwin && w0 + mwin < nwin_total) {
            const int64_t widx = window_index(a.pg, a.Hkv, a.t_cap, b, h, w0 + mwin, bad_page);
            ms0 = a.kms[widx];
            mv0 = *reinterpret_cast<const uint32_t*>(a.kmq + widx * kD + 4 * (lane & 31));
        }
    }
    const int T = min(a.seq_lens[b], a.t_cap);
    if (start >= T) return;   // the merge ignores chunks past the length
    const int ntiles = (min(a.chunk, T - start) + kTile - 1) / kTile;
    // windows from the sequence's length on are never used
    auto mean_live = [&](int wi) {
        return wi < nwin && w0 + wi < nwin_total && (w0 + wi) * DQ_MEAN_WINDOW < T;
    };
    if (paged) {
        if (kPrefetch) {
            const int ft = min(ptile, ntiles - 1);
            const int64_t tok = record_row(a.pg, a.Hkv, a.t_cap, b, h, start + ft * kTile, bad_page) + lane;
            if (load_k) load_record(rk, a.krec, tok, CWk);
            if (load_v) load_record(rv, a.vrec, tok, CWv);
            else rv[0] = *reinterpret_cast<const uint32_t*>(a.vrec + tok * (CWv * 4));
        }
        if (mean_live(mwin)) {
            const int64_t widx = window_index(a.pg, a.Hkv, a.t_cap, b, h, w0 + mwin, bad_page);
            ms0 = a.kms[widx];
            mv0 = *reinterpret_cast<const uint32_t*>(a.kmq + widx * kD + 4 * (lane & 31));
        }
    }

    // ---- prologue: tables, rotated query, its digits, q . mu per window
    if (!FIXED && wave >= tw0) {
        stage_store(reinterpret_cast<uint2*>(smem + L.lut_k), lut_e, Pk, ttid, tthr);
        stage_table(reinterpret_cast<uint2*>(smem + L.lut_k), a.tk.t.lut64, Pk, ttid, tthr);
        if (LUTV != 0) {
            stage_store(reinterpret_cast<uint2*>(smem + LUTV), lutv_e, Pv, ttid, tthr);
            stage_table(reinterpret_cast<uint2*>(smem + LUTV), a.tv.t.lut64, Pv, ttid, tthr);
        }
    }
    float* qt = reinterpret_cast<float*>(smem + L.waves);          // [G][d] scratch
    float* qscale = reinterpret_cast<float*>(smem + L.qscale);
    float* qsum = reinterpret_cast<float*>(smem + L.qsum);
    float* qmu = reinterpret_cast<float*>(smem + L.qmu);
    uint8_t* qlimb = smem + L.qlimb;
    // wavefront g rotates query head g and forms its digits from the
    // registers (slots past G get zero digits); a workgroup with fewer
    // wavefronts than head slots loads the other heads here, the first head
    // of a wavefront needs no wait on the records
    auto head_digits = [&](float r0, float r1, float qs, int g) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int j = lane + 64 * hh;
            int v = 0;
            if (qs > 0.f) {
                v = (int)rintf((hh ? r1 : r0) / qs);
                v = max(-4194304, min(4194304, v));
            }
            int d0, d1, d2;
            digits3(v, d0, d1, d2);
            uint8_t* dst = qlimb + ((j / 4) * GP + g) * 16 + (j % 4);
            dst[0] = (uint8_t)d0;
            dst[4] = (uint8_t)d1;
            dst[8] = (uint8_t)d2;
            dst[12] = 0;
        }
    };
    if (wave < G) {
        // consumed here, not where loaded: a wait there would hold back the
        // loads behind it
        uint32_t w0 = qb0, w1 = qb1;
        asm volatile("" : "+v"(w0), "+v"(w1));
        float v0 = bf16_to_f32((uint16_t)w0), v1 = bf16_to_f32((uint16_t)w1);
        const float qs = rotate_query_head(v0, v1, wave, lane, qt, qscale, qsum, a.rot_q);
        head_digits(v0, v1, qs, wave);
    } else if (wave < GP) {
        if (lane == 0) qscale[wave] = qsum[wave] = 0.f;
        head_digits(0.f, 0.f, 0.f, wave);
    }
    for (int g = wave + L.nw; g < GP; g += L.nw) {
        if (g >= G) {
            if (lane == 0) qscale[g] = qsum[g] = 0.f;
            head_digits(0.f, 0.f, 0.f, g);
            continue;
        }
        const uint16_t* qh = a.q + ((int64_t)b * a.Hq + hq0 + g) * kD;
        float v0 = bf16_to_f32(qh[lane]), v1 = bf16_to_f32(qh[lane + 64]);
        const float qs = rotate_query_head(v0, v1, g, lane, qt, qscale, qsum, a.rot_q);
        head_digits(v0, v1, qs, g);
    }
    __syncthreads();
    {
        const int r = lane >> 5, c4 = 4 * (lane & 31);
        for (int wi = 2 * mwave + r, pass = 0; wi - r < nwin; wi += 2 * L.nw, ++pass) {
            float f[4] = {0.f, 0.f, 0.f, 0.f};
            if (mean_live(wi)) {
                uint32_t mv = mv0;
                uint16_t ms = ms0;
                if (pass > 0) {
                    const int64_t widx = window_index(a.pg, a.Hkv, a.t_cap, b, h, w0 + wi, bad_page);
                    ms = a.kms[widx];
                    mv = *reinterpret_cast<const uint32_t*>(a.kmq + widx * kD + c4);
                }
                const float sc = half_bits_to_f32(ms);
#pragma unroll
                for (int k = 0; k < 4; ++k) f[k] = sc * (float)(int8_t)((mv >> (8 * k)) & 0xFF);
            }
            // every head slot at once, without branches (rows of slots past G
            // hold no query: their sums are replaced by 0), so that the LDS
            // reads and the half-wavefront sums of the slots overlap
            float sg[GP];
#pragma unroll
            for (int g = 0; g < GP; ++g) {
                const float4 qv = *reinterpret_cast<const float4*>(qt + g * kD + c4);
                float s = 0.f;
                s = s + qv.x * f[0];
                s = s + qv.y * f[1];
                s = s + qv.z * f[2];
                s = s + qv.w * f[3];
                sg[g] = s;
            }
#pragma unroll
            for (int g = 0; g < GP; ++g) sg[g] = half_sum_f32(sg[g]);
            if ((lane & 31) == 31 && wi < nwin) {
#pragma unroll
                for (int g = 0; g < GP; ++g) qmu[wi * GP + g] = g < G ? sg[g] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- per-wavefront state
    uint8_t* wreg = smem + L.waves + wave * L.wave_stride;
    // lane l's column in a row of 64 pairs: lanes l and l + 32 share a dword,
    // so each half-wavefront reads 32 different banks
    const uint32_t col = (uint32_t)(4 * (lane & 31) + 2 * (lane >> 5));
    const uint32_t pk_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.pk) + col;
    const uint32_t pv_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.pv) + col;
    uint8_t* vtile = wreg + L.vtile;     // overlays the pair arrays once both streams are decoded
    uint8_t* plimb = wreg + L.plimb;
    // P . v: lane l serves query-head slot l / 16 and channel l % 16 of each
    // 16-channel block; its tr8 reads start at token row 8 (l / 16) +
    // (l % 16) / 2 of a 32-token block, byte 8 (l % 2) of the row's block
    const int slot = lane >> 4;
    const uint32_t trow = (uint32_t)(8 * (lane >> 4) + ((lane & 15) >> 1));
    const uint32_t a_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.plimb) + trow * 16 + 8 * (lane & 1);
    const uint32_t b_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.vtile) + trow * kVRowT + 8 * (lane & 1);
    const int pk3 = a.tk.p + 3, pv3 = a.tv.p + 3;
    const uint32_t mask8k = ((1u << a.tk.p) - 1u) << 3, mask8v = ((1u << a.tv.p) - 1u) << 3;
    const int64_t bh = (int64_t)b * a.Hkv + h;

    // softmax state per query head (the same in every lane); the P . v sums
    // of slot l / 16 of group hg, channel 64 s + 16 cb + l % 16 in acc[s][hg][cb]
    float m_run[GP], l_part[GP], acco[GP], acc[2][HG][4];
#pragma unroll
    for (int g = 0; g < GP; ++g) {
        m_run[g] = -INFINITY;
        l_part[g] = 0.f;
        acco[g] = 0.f;
    }
#pragma unroll
    for (int hg = 0; hg < HG; ++hg)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) acc[0][hg][cb] = acc[1][hg][cb] = 0.f;
    bool corrupt = false;
    float l_tot[GP], o_tot[GP];

    if constexpr (SPLIT) {
        // One tile per pair of wavefronts: the even wavefront decodes the
        // keys, forms the scores and the softmax weights and leaves their
        // digits (its weight-digit tile) and the tile's statistics in its LDS
        // region; the odd one decodes the values meanwhile and, after the
        // barrier, forms P . v with its partner's weights.  Each chain then
        // has its SIMD to itself: a step waits only for its own two LDS reads
        // (two chains in one wavefront take a third longer per tile, which
        // bounds the latency when one wavefront runs per SIMD).
        static_assert(HG == 1 && !FIXED, "split tiles: up to 4 query heads, entropy-coded records");
        const int tile = wave >> 1, role = wave & 1;
        // [0, GP) weight scale of each slot, then maxima, sums, offset sums
        float* kx = reinterpret_cast<float*>(smem + L.waves + (wave & ~1) * L.wave_stride + L.vtile);
        uint32_t vlev[kD / 4];
        const int t_base = start + tile * kTile;
        const int t = t_base + lane;
        const bool valid = t < T;
        uint32_t rr_;
        uint64_t ee_;
        if (tile < ntiles && role == 0) {
            const uint32_t hk0 = rk[0], hv0 = rv[0];
            uint32_t xk = rk[1] << 3;
            build_pairs(rk, CWk, smem + pk_lane);
            asm volatile("" ::: "memory");
            uint32_t pq = pk_lane;
            const uint32_t pk_end = pk_lane + (uint32_t)((Ck - kPayloadOffset) * kPairRow);
            v4i dk[3];
#pragma unroll
            for (int d = 0; d < 3; ++d) dk[d] = v4i{0, 0, 0, 0};
            const uint32_t q_lane = (uint32_t)L.qlimb + (uint32_t)(lane & 3) * 16;
            v4u qd;
            dissue<0>(xk, pq, mask8k, 0, rr_, ee_);
#pragma unroll
            for (int grp = 0; grp < kD / 4; ++grp) {
                uint32_t kw[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int n = 4 * grp + u, J1 = (n + 1) % kWindow;
                    const bool more = n + 1 < kD;
                    dwait<0>(rr_, ee_);
                    kw[u] = dfinish(xk, pq, pk3, rr_, ee_);
                    if (J1 == 0) {
                        pq += kWindow * kPairStep;
                        if (more) pq = min(pq, pk_end);
                    }
                    if (u == 3) qissue(q_lane, (grp * GP) * 16, qd);
                    if (more) dissue<0>(xk, pq, mask8k, J1, rr_, ee_);
                }
                const uint32_t lk = pack4(kw[0], kw[1], kw[2], kw[3]);
                // the digits were requested before the next step's two reads
                if (grp + 1 < kD / 4) dwaitq1<2>(qd);
                else dwaitq1<0>(qd);
                dk[0] = mfma(qd.x, lk, dk[0]);
                dk[1] = mfma(qd.y, lk, dk[1]);
                dk[2] = mfma(qd.z, lk, dk[2]);
                __builtin_amdgcn_sched_barrier(0);
            }
            corrupt |= valid && ((xk >> 3) != kRansL || pq > pk_end);
            // scores (Eq. fold-key) and the tile's softmax; the value scale is
            // folded into the weight (Eq. fold-value)
            const float sk = half_lo(hk0), ok = half_hi(hk0);
            const float sv = half_lo(hv0), ov = half_hi(hv0);
            const float* qm = qmu + ((t / DQ_MEAN_WINDOW) - w0) * GP;
            float score[4], tmax[4], pw[4], smax[4], lp[4], op[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float dot = combine(dk[0], dk[1], dk[2], r) * qscale[r];
                score[r] = (valid && r < G) ? (sk * dot + ok * qsum[r] + qm[r]) * a.scale_log2 : -INFINITY;
                tmax[r] = score[r];
            }
            wave_max4_f32(tmax);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float p = (score[r] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(score[r] - tmax[r]);
                lp[r] = p;
                op[r] = p * ov;
                pw[r] = p * sv;
                smax[r] = pw[r];
            }
            wave_max4_f32(smax);
            uint32_t wd[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float inv = smax[r] > 0.f ? 4194304.0f * __builtin_amdgcn_rcpf(smax[r]) : 0.f;
                const int pint = min(4194304, (int)rintf(pw[r] * inv));
                int d0, d1, d2;
                digits3(pint, d0, d1, d2);
                wd[r] = ((uint32_t)d0 & 0xFFu) | (((uint32_t)d1 & 0xFFu) << 8) | (((uint32_t)d2 & 0xFFu) << 16);
                l_tot[r] = wave_sum_f32(lp[r]);
                o_tot[r] = wave_sum_f32(op[r]);
            }
            *reinterpret_cast<uint4*>(plimb + lane * 16) = uint4{wd[0], wd[1], wd[2], wd[3]};
            if (lane == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    kx[r] = smax[r] * (1.0f / 4194304.0f);
                    kx[GP + r] = tmax[r];
                    kx[2 * GP + r] = l_tot[r];
                    kx[3 * GP + r] = o_tot[r];
                }
            }
        } else if (tile < ntiles) {
            uint32_t xv = rv[1] << 3;
            build_pairs(rv, CWv, smem + pv_lane);
            asm volatile("" ::: "memory");
            uint32_t pv = pv_lane;
            const uint32_t pv_end = pv_lane + (uint32_t)((Cv - kPayloadOffset) * kPairRow);
            dissue<LUTV>(xv, pv, mask8v, 0, rr_, ee_);
#pragma unroll
            for (int grp = 0; grp < kD / 4; ++grp) {
                uint32_t vw[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int n = 4 * grp + u, J1 = (n + 1) % kWindow;
                    const bool more = n + 1 < kD;
                    dwait<0>(rr_, ee_);
                    vw[u] = dfinish(xv, pv, pv3, rr_, ee_);
                    if (J1 == 0) {
                        pv += kWindow * kPairStep;
                        if (more) pv = min(pv, pv_end);
                    }
                    if (more) dissue<LUTV>(xv, pv, mask8v, J1, rr_, ee_);
                }
                vlev[grp] = pack4(vw[0], vw[1], vw[2], vw[3]);
                asm volatile("" : "+v"(vlev[grp]));
                __builtin_amdgcn_sched_barrier(0);
            }
            corrupt |= valid && ((xv >> 3) != kRansL || pv > pv_end);
        }
        __syncthreads();   // the weights and statistics of every pair are in LDS
        if (tile < ntiles && role == 1) {
            // ---- P . v with the partner's weight digits, two slices of 64 channels
            const uint32_t a_pair = a_lane - (uint32_t)L.wave_stride;
            uint64_t pa[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) pa[kb] = lds_tr8(a_pair + kb * 32 * 16);
            const float scale_l = pick4(kx, slot);
#pragma unroll
            for (int g = 0; g < GP; ++g) {
                m_run[g] = kx[GP + g];
                l_tot[g] = kx[2 * GP + g];
                o_tot[g] = kx[3 * GP + g];
            }
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                if (sl) wave_sync();   // the first slice's value rows are no longer read
#pragma unroll
                for (int qq = 0; qq < 4; ++qq)
                    *reinterpret_cast<uint4*>(vtile + lane * kVRowT + 16 * qq) =
                        uint4{vlev[16 * sl + 4 * qq], vlev[16 * sl + 4 * qq + 1], vlev[16 * sl + 4 * qq + 2],
                              vlev[16 * sl + 4 * qq + 3]};
                wave_sync();
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    const uint64_t b0 = lds_tr8(b_lane + 16 * cb);
                    const uint64_t b1 = lds_tr8(b_lane + 32 * kVRowT + 16 * cb);
                    v4i d = mfma16(pa[0], b0, v4i{0, 0, 0, 0});
                    d = mfma16(pa[1], b1, d);
                    acc[sl][0][cb] = ((float)d[2] * 65536.0f + (float)d[1] * 256.0f + (float)d[0]) * scale_l;
                }
            }
        }
    }

    for (int tile = SPLIT ? ntiles : wave; tile < ntiles; tile += L.nw) {
        const int t_base = start + tile * kTile;
        const int t = t_base + lane;
        const bool valid = t < T;
        if (!kPrefetch) {
            const int64_t tok = record_row(a.pg, a.Hkv, a.t_cap, b, h, t_base, bad_page) + lane;
            load_record(rk, a.krec, tok, CWk);
            load_record(rv, a.vrec, tok, CWv);
        }

        // ---- both records of the lane's token -> headers + byte-pair arrays
        const uint32_t hk0 = rk[0], xk0 = rk[1] << 3;
        const uint32_t hv0 = rv[0], xv0 = rv[1] << 3;
        uint32_t ck[FIXED ? 9 : 1], cv[FIXED ? 9 : 1];   // this tile's fixed-width records
        if (FIXED) {
#pragma unroll
            for (int k = 0; k < (FIXED ? 9 : 1); ++k) {
                ck[k] = rk[k];
                cv[k] = rv[k];
            }
        } else {
            build_pairs(rk, CWk, smem + pk_lane);
            build_pairs(rv, CWv, smem + pv_lane);
        }
        uint32_t xk = xk0, xv = xv0;
        // the pair arrays are read back by this lane only: order the reads
        // after the writes (LDS keeps a wavefront's accesses in order)
        asm volatile("" ::: "memory");
        uint32_t pq = pk_lane, pv = pv_lane;
        // one past the last payload position: a valid stream never reads beyond
        const uint32_t pk_end = pk_lane + (uint32_t)((Ck - kPayloadOffset) * kPairRow);
        const uint32_t pv_end = pv_lane + (uint32_t)((Cv - kPayloadOffset) * kPairRow);

        // ---- keys and values decoded together: two independent rANS chains
        //      per lane.  Key levels go straight into the q . k products; value
        //      levels wait in registers until the softmax weights are known.
        v4i dk[HG][3];
#pragma unroll
        for (int hg = 0; hg < HG; ++hg)
#pragma unroll
            for (int d = 0; d < 3; ++d) dk[hg][d] = v4i{0, 0, 0, 0};
        uint32_t vlev[kD / 4];
        // the query digits of group g are requested after the key step 4 g + 3,
        // so that the wait for the value step 4 g + 3 covers them too
        const uint32_t q_lane = (uint32_t)L.qlimb + (uint32_t)(lane & 3) * 16;
        v4u qd[HG];
        // step n of both chains: wait for its reads, finish it, request step
        // n + 1 (pointer windows advance and are clamped between n and n + 1;
        // a corrupt stream may run past its array, so clamp often enough
        // that it cannot leave the workgroup's LDS (kPairSlack above the
        // arrays), except after the last window, whose pointer is checked)
        uint32_t rk_, rv_;
        uint64_t ek_, ev_;
        if (!FIXED) {
            dissue<0>(xk, pq, mask8k, 0, rk_, ek_);
            dissue<LUTV>(xv, pv, mask8v, 0, rv_, ev_);
        }
        // A wavefront in the decode runs at a raised priority: its two
        // dependent chains issue first whenever they are ready, and the
        // softmax, P . v and pair building of the other wavefronts, which have
        // more independent work, fill the slots in between (7 % less time at
        // 16 wavefronts than at one priority for all).
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int grp = 0; grp < kD / 4; ++grp) {
            uint32_t lk;
            if (FIXED) {
                const int w = 1 + (FIXED ? grp / 4 : 0), sh = 8 * (grp % 4);
                lk = spread2(__builtin_amdgcn_ubfe(ck[w], sh, 8));
                vlev[grp] = spread2(__builtin_amdgcn_ubfe(cv[w], sh, 8));
#pragma unroll
                for (int hg = 0; hg < HG; ++hg)
                    qd[hg] = *reinterpret_cast<const v4u*>(qlimb + ((grp * GP) + hg * 4 + (lane & 3)) * 16);
            } else {
                uint32_t kw[4], vw[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int n = 4 * grp + u, J1 = (n + 1) % kWindow;
                    const bool more = n + 1 < kD;
                    dwait<2>(rk_, ek_);                  // the value reads of step n follow
                    kw[u] = dfinish(xk, pq, pk3, rk_, ek_);
                    if (J1 == 0) {
                        pq += kWindow * kPairStep;
                        if (more) pq = min(pq, pk_end);
                    }
                    if (u == 3) {
                        qissue(q_lane, (grp * GP) * 16, qd[0]);
                        if constexpr (HG == 2) qissue(q_lane, (grp * GP + 4) * 16, qd[1]);
                    }
                    if (more) dissue<0>(xk, pq, mask8k, J1, rk_, ek_);
                    // the key reads of step n + 1 follow (and the digits at u = 3,
                    // before them: this wait covers those too)
                    if (u < 3) dwait<2>(rv_, ev_);
                    else if (more) dwaitq<2>(rv_, ev_, qd);
                    else dwaitq<0>(rv_, ev_, qd);
                    vw[u] = dfinish(xv, pv, pv3, rv_, ev_);
                    if (J1 == 0) {
                        pv += kWindow * kPairStep;
                        if (more) pv = min(pv, pv_end);
                    }
                    if (more) dissue<LUTV>(xv, pv, mask8v, J1, rv_, ev_);
                }
                lk = pack4(kw[0], kw[1], kw[2], kw[3]);
                vlev[grp] = pack4(vw[0], vw[1], vw[2], vw[3]);
            }
            // pack now: left alone, the packing sinks to the value pass and the
            // four table words stay live until then
            asm volatile("" : "+v"(vlev[grp]));
#pragma unroll
            for (int hg = 0; hg < HG; ++hg) {
                dk[hg][0] = mfma(qd[hg].x, lk, dk[hg][0]);
                dk[hg][1] = mfma(qd[hg].y, lk, dk[hg][1]);
                dk[hg][2] = mfma(qd[hg].z, lk, dk[hg][2]);
            }
            // keep the scheduler inside one group: live ranges stay short
            __builtin_amdgcn_sched_barrier(0);
        }
        // every stream ends at x = L having read at most its C - 8 payload bytes
        if (!FIXED) {
            corrupt |= valid && ((xk >> 3) != kRansL || pq > pk_end);
            corrupt |= valid && ((xv >> 3) != kRansL || pv > pv_end);
        }

        __builtin_amdgcn_s_setprio(0);
        // ---- scores (Eq. fold-key) and online softmax; the value scale is
        //      folded into the weight (Eq. fold-value)
        const float sk = half_lo(hk0), ok = half_hi(hk0);
        const float sv = half_lo(hv0), ov = half_hi(hv0);
        const float* qm = qmu + ((t / DQ_MEAN_WINDOW) - w0) * GP;
        float pscale[GP], corrs[GP];
        int pint[GP];
        // four query heads at a time, their tile maxima reduced together
#pragma unroll
        for (int hg = 0; hg < HG; ++hg) {
            float score[4], tmax[4], pw[4], smax[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int g = 4 * hg + r;
                const float dot = combine(dk[hg][0], dk[hg][1], dk[hg][2], r) * qscale[g];
                score[r] = (valid && g < G) ? (sk * dot + ok * qsum[g] + qm[g]) * a.scale_log2 : -INFINITY;
                tmax[r] = score[r];
            }
            wave_max4_f32(tmax);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int g = 4 * hg + r;
                const float mn = fmaxf(m_run[g], tmax[r]);
                // v_exp_f32 directly: arguments are <= 0 and results that would
                // be denormal may flush to zero
                const float corr = (m_run[g] == -INFINITY || mn == -INFINITY) ? (m_run[g] == mn ? 1.f : 0.f)
                                                                               : __builtin_amdgcn_exp2f(m_run[g] - mn);
                const float p = (score[r] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(score[r] - mn);
                l_part[g] = l_part[g] * corr + p;
                acco[g] = acco[g] * corr + p * ov;
                corrs[g] = corr;
                m_run[g] = mn;
                pw[r] = p * sv;                          // >= 0: scales are non-negative
                smax[r] = pw[r];
            }
            wave_max4_f32(smax);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int g = 4 * hg + r;
                pscale[g] = smax[r] * (1.0f / 4194304.0f);
                // 22-bit fixed point of pw relative to the tile maximum
                const float inv = smax[r] > 0.f ? 4194304.0f * __builtin_amdgcn_rcpf(smax[r]) : 0.f;
                pint[g] = min(4194304, (int)rintf(pw[r] * inv));
            }
        }
        // weight digits -> LDS, one 16-byte token row per slot group: byte
        // 4 r + d holds digit d of slot r (byte 4 r + 3 stays zero)
#pragma unroll
        for (int hg = 0; hg < HG; ++hg) {
            uint32_t w[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int d0, d1, d2;
                digits3(pint[4 * hg + r], d0, d1, d2);
                w[r] = ((uint32_t)d0 & 0xFFu) | (((uint32_t)d1 & 0xFFu) << 8) | (((uint32_t)d2 & 0xFFu) << 16);
            }
            *reinterpret_cast<uint4*>(plimb + hg * (kTile * 16) + lane * 16) = uint4{w[0], w[1], w[2], w[3]};
        }
        float scale_l[HG];
#pragma unroll
        for (int hg = 0; hg < HG; ++hg) {
            const float corr_l = pick4(corrs + 4 * hg, slot);
            scale_l[hg] = pick4(pscale + 4 * hg, slot);
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                acc[0][hg][cb] *= corr_l;
                acc[1][hg][cb] *= corr_l;
            }
        }

        if (kPrefetch && tile + L.nw < ntiles) {
            const int64_t tok = record_row(a.pg, a.Hkv, a.t_cap, b, h, t_base + L.nw * kTile, bad_page) + lane;
            load_record(rk, a.krec, tok, CWk);
            load_record(rv, a.vrec, tok, CWv);
        }

        // ---- P . v over two slices of 64 channels
        wave_sync();   // the weight rows (and, below, the value rows) are read by other lanes
        uint64_t pa[HG][2];
#pragma unroll
        for (int hg = 0; hg < HG; ++hg)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) pa[hg][kb] = lds_tr8(a_lane + hg * (kTile * 16) + kb * 32 * 16);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            if (s) wave_sync();   // the first slice's value rows are no longer read
            // the lane's 64 levels of the slice: 4 x 16 bytes of its token row
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<uint4*>(vtile + lane * kVRowT + 16 * q) =
                    uint4{vlev[16 * s + 4 * q], vlev[16 * s + 4 * q + 1], vlev[16 * s + 4 * q + 2],
                          vlev[16 * s + 4 * q + 3]};
            wave_sync();
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const uint64_t b0 = lds_tr8(b_lane + 16 * cb);
                const uint64_t b1 = lds_tr8(b_lane + 32 * kVRowT + 16 * cb);
#pragma unroll
                for (int hg = 0; hg < HG; ++hg) {
                    v4i d = mfma16(pa[hg][0], b0, v4i{0, 0, 0, 0});
                    d = mfma16(pa[hg][1], b1, d);
                    acc[s][hg][cb] += ((float)d[2] * 65536.0f + (float)d[1] * 256.0f + (float)d[0]) * scale_l[hg];
                }
            }
        }
        wave_sync();   // the next tile rewrites the pair arrays over the value tile
    }
    if (__any(corrupt) && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_CORRUPT);
    if (__any(bad_page) && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_PAGE);

    // ---- merge the wavefronts of the workgroup (SPLIT: the pairs, whose
    //      statistics the value wavefront has read from its partner)
    if constexpr (!SPLIT) {
#pragma unroll
        for (int g = 0; g < GP; ++g) {
            l_tot[g] = wave_sum_f32(l_part[g]);
            o_tot[g] = wave_sum_f32(acco[g]);
        }
    }
    __syncthreads();   // every wavefront is done with LDS
    float* mw = reinterpret_cast<float*>(smem);        // [nw][GP]
    float* lw = mw + L.nw * GP;                        // [nw][GP]
    float* aw = lw + L.nw * GP;                        // [nw][GP][d]
    if (!SPLIT || ((wave & 1) && (wave >> 1) < ntiles)) {
        const int ws = SPLIT ? wave >> 1 : wave;
#pragma unroll
        for (int g = 0; g < GP; ++g) {
            if (lane == 0) {
                mw[ws * GP + g] = m_run[g];
                lw[ws * GP + g] = l_tot[g];
            }
        }
#pragma unroll
        for (int hg = 0; hg < HG; ++hg) {
            const float o_l = pick4(o_tot + 4 * hg, slot);
            float* row = aw + (ws * GP + 4 * hg + slot) * kD + (lane & 15);
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                row[16 * cb] = acc[0][hg][cb] + o_l;
                row[kVSlice + 16 * cb] = acc[1][hg][cb] + o_l;
            }
        }
    }
    __syncthreads();
    const int NC = a.nchunks;
    // only the wavefronts that decoded a tile hold partials; they are read in
    // blocks of four whose loads are in flight together (indexes clamped)
    const int nwa = min(L.nw, ntiles);
    for (int i = tid; i < G * kD; i += nthr) {
        const int g = i / kD, j = i % kD;
        float M = -INFINITY;
        for (int w0 = 0; w0 < nwa; w0 += 4) {
#pragma unroll
            for (int u = 0; u < 4; ++u) M = fmaxf(M, mw[min(w0 + u, nwa - 1) * GP + g]);
        }
        float acc = 0.f, l = 0.f;
        for (int w0 = 0; w0 < nwa; w0 += 4) {
            float mv[4], av[4], lv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int ww = min(w0 + u, nwa - 1);
                mv[u] = mw[ww * GP + g];
                av[u] = aw[(ww * GP + g) * kD + j];
                lv[u] = lw[ww * GP + g];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (w0 + u >= nwa || mv[u] == -INFINITY) continue;
                const float e = exp2f(mv[u] - M);
                acc += av[u] * e;
                l += lv[u] * e;
            }
        }
        const int64_t slot = ((int64_t)b * a.Hq + hq0 + g) * (NC + kResSlots) + c;
        a.ws_acc[slot * kD + j] = acc;
        if (j == 0) {
            a.ws_m[slot] = M;
            a.ws_l[slot] = l;
        }
    }
}

// One wavefront per (query head, sequence): lane l combines channels l and
// l + 64 of every partial, so no barrier is needed anywhere.  Lane i holds
// the maximum and sum of partial i (of the first 64); the accumulator rows
// of up to kMergeBatch partials are requested together with them, right
// after the header: one memory round trip for the usual counts (b1_t128k: 32
// chunks + 4 residual slots), a further one per batch beyond.
constexpr int kMergeBatch = 32;

__global__ __launch_bounds__(kWave) void attn_merge_kernel(const int32_t* __restrict__ ws_hdr,
                                                           const float* __restrict__ ws_m,
                                                           const float* __restrict__ ws_l,
                                                           const float* __restrict__ ws_acc,
                                                           const int32_t* __restrict__ seq_lens,
                                                           int Hq, int t_cap, int nc_max, float* __restrict__ out) {
    const int hq = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
    // the header's chunk count is bounded by the workspace's capacity, so a
    // workspace no partial call wrote cannot send the reads past it
    const int chunk = max(ws_hdr[0], 1), NC = min(max(ws_hdr[1], 1), nc_max);
    const int residual = min(max(ws_hdr[2], 0), kResSlots);
    const int T = max(0, min(seq_lens[b], t_cap));
    float* dst = out + ((int64_t)b * Hq + hq) * kD;
    // the chunks that hold tokens, then the residual window's slots (a part
    // of the window without tokens wrote m = -inf)
    const int nc = min(NC, (T + chunk - 1) / chunk);
    const int64_t base = ((int64_t)b * Hq + hq) * (NC + kResSlots);
    // partials in use: chunks 0..nc-1, then the residual slots NC..
    const int np = nc + residual;
    auto slot_of = [&](int i) { return base + (i < nc ? i : NC + i - nc); };
    if (np == 0) {
        dst[lane] = 0.f;
        dst[lane + 64] = 0.f;
        return;
    }
    // every load of the first round at once (indexes clamped: unconditional)
    const int64_t sl = slot_of(min(lane, np - 1));
    const float m_lane = lane < np ? ws_m[sl] : -INFINITY;
    const float l_lane = lane < np ? ws_l[sl] : 0.f;
    float a0[kMergeBatch], a1[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
        const int64_t s = slot_of(min(u, np - 1));
        a0[u] = ws_acc[s * kD + lane];
        a1[u] = ws_acc[s * kD + lane + 64];
    }
    float M = m_lane;
    for (int i = lane + kWave; i < np; i += kWave) M = fmaxf(M, ws_m[slot_of(i)]);
    M = wave_max_f32(M);
    if (M == -INFINITY) {      // no token at all
        dst[lane] = 0.f;
        dst[lane + 64] = 0.f;
        return;
    }
    // weight of partial i: lane i for the first 64, computed in place beyond
    const float e_lane = lane < np ? exp2f(m_lane - M) : 0.f;
    float l = wave_sum_f32(l_lane * e_lane);
    float acc0 = 0.f, acc1 = 0.f;
    for (int i0 = 0;;) {
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const int i = i0 + u;
            float e = 0.f;
            if (i < np) {
                if (i < kWave) {
                    e = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(e_lane), i));
                } else {
                    const int64_t s = slot_of(i);
                    e = exp2f(ws_m[s] - M);
                    l += ws_l[s] * e;
                }
            }
            acc0 += a0[u] * e;
            acc1 += a1[u] * e;
        }
        i0 += kMergeBatch;
        if (i0 >= np) break;
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const int64_t s = slot_of(min(i0 + u, np - 1));
            a0[u] = ws_acc[s * kD + lane];
            a1[u] = ws_acc[s * kD + lane + 64];
        }
    }
    float v0 = acc0 / l, v1 = acc1 / l;
    if (ws_hdr[3]) {           // inverse rotation of the value basis: H v / d
        hadamard_lanes(v0, v1, lane);
        const float r0 = (v0 + v1) * (1.0f / kD), r1 = (v0 - v1) * (1.0f / kD);
        v0 = r0;
        v1 = r1;
    }
    dst[lane] = v0;
    dst[lane + 64] = v1;
}

// ------------------------------------------------------- residual window
//
// The most recent tokens of a sequence stay in bf16 (Sec. 5.1).  They live in
// a ring of r_cap slots per (sequence, KV head): residual token i of sequence
// b is slot (seq_lens[b] + i) mod r_cap, so the oldest tokens are contiguous
// whenever the compressed length is a multiple of the window being flushed.

constexpr int kResThreads = 256;
constexpr int kMaxResidual = 256;
constexpr int kMaxGroup = 8;
constexpr int kResWaves = 2;                          // wavefronts per part
constexpr int kResWaveTokens = kMaxResidual / kResSlots / kResWaves;   // at most 32 per wavefront

struct ResArgs {
    const uint16_t* q;
    const uint16_t* rk;          // [B][Hkv][r_cap][d] bf16
    const uint16_t* rv;
    const int32_t* seq_lens;     // compressed tokens per sequence
    const int32_t* res_lens;     // residual tokens per sequence
    int r_cap, Hq, Hkv, G;
    float scale_log2;            // softmax_scale * log2(e): logits of raw keys
    int nc_max;                  // chunk slots per query head the workspace holds
    int32_t* ws_hdr;
    float* ws_m;
    float* ws_l;
    float* ws_acc;
};

// Maximum and sum over each row of 16 lanes; every lane of the row ends with
// the row's result.
__device__ __forceinline__ float row_max_f32(float v) {
    v = fmaxf(v, dpp_step<0xB1, 0xF>(v));    // quad_perm [1, 0, 3, 2]
    v = fmaxf(v, dpp_step<0x4E, 0xF>(v));    // quad_perm [2, 3, 0, 1]
    v = fmaxf(v, dpp_step<0x141, 0xF>(v));   // row_half_mirror
    return fmaxf(v, dpp_step<0x140, 0xF>(v));   // row_mirror
}
__device__ __forceinline__ float row_sum_f32(float v) {
    v += dpp_step<0xB1, 0xF>(v);
    v += dpp_step<0x4E, 0xF>(v);
    v += dpp_step<0x141, 0xF>(v);
    return v + dpp_step<0x140, 0xF>(v);
}

// bf16 pairs a . b + c in fp32 (v_dot2c_f32_bf16)
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}

// Softmax partial of nw <= NT raw tokens (ring positions ring0 + i, wrapping
// at r_cap) for the G query heads of KV head h, in one wavefront:
// * logits: lane l takes tokens l % 16 (+ 16) and channels 32 (l / 16) .. + 31,
//   bf16 pair products summed in fp32, then summed over the four rows with
//   lane swaps; every row then holds every logit;
// * statistics per head over the row (DPP), weights to p_lds[g][token];
// * values: lane l takes channels 2 l and 2 l + 1 of every token and the
//   weights from LDS (one broadcast read per 4 tokens and head).
// Every load is requested before the first is used (one memory round trip).
template <int NT>
__device__ __forceinline__ void residual_wave(const ResArgs& a, int b, int h, int ring0, int nw, int lane,
                                              float (*p_lds)[kResWaveTokens], float (&acc)[kMaxGroup][2],
                                              float (&mx)[kMaxGroup], float (&sm)[kMaxGroup]) {
    constexpr int NS = NT / 16;
    const int G = a.G, ti = lane & 15, cq = lane >> 4;
    const int64_t row0 = ((int64_t)b * a.Hkv + h) * a.r_cap;
    auto row = [&](int i) {           // ring slot of token min(i, nw - 1) (ring0 + i < 2 r_cap)
        const int s = ring0 + min(i, nw - 1);
        return row0 + (s < a.r_cap ? s : s - a.r_cap);
    };
    uint4 kr[NS][4];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const uint4* src = reinterpret_cast<const uint4*>(a.rk + row(ti + 16 * j) * kD + 32 * cq);
#pragma unroll
        for (int u = 0; u < 4; ++u) kr[j][u] = src[u];
    }
    uint4 qr[kMaxGroup][4];
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) {
        if (g < G) {
            const uint4* src = reinterpret_cast<const uint4*>(a.q + ((int64_t)b * a.Hq + h * G + g) * kD + 32 * cq);
#pragma unroll
            for (int u = 0; u < 4; ++u) qr[g][u] = src[u];
        }
    }
    uint32_t vr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) vr[t] = *reinterpret_cast<const uint32_t*>(a.rv + row(t) * kD + 2 * lane);

#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) {
        if (g < G) {
            float s[NS];
#pragma unroll
            for (int j = 0; j < NS; ++j) {
                float d = 0.f;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    d = dot2_bf16(qr[g][u].x, kr[j][u].x, d);
                    d = dot2_bf16(qr[g][u].y, kr[j][u].y, d);
                    d = dot2_bf16(qr[g][u].z, kr[j][u].z, d);
                    d = dot2_bf16(qr[g][u].w, kr[j][u].w, d);
                }
                d += xor_lane<16>(d, lane);
                d += xor_lane<32>(d, lane);
                s[j] = ti + 16 * j < nw ? d * a.scale_log2 : -INFINITY;
            }
            float m = s[0];
#pragma unroll
            for (int j = 1; j < NS; ++j) m = fmaxf(m, s[j]);
            m = row_max_f32(m);
            float l = 0.f;
#pragma unroll
            for (int j = 0; j < NS; ++j) {
                s[j] = exp2f(s[j] - m);
                l += s[j];
                if (cq == 0) p_lds[g][ti + 16 * j] = s[j];
            }
            mx[g] = m;
            sm[g] = row_sum_f32(l);
        }
    }
    // the weights were written by lanes of this wavefront, whose LDS
    // operations complete in order
    wave_sync();
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) acc[g][0] = acc[g][1] = 0.f;
#pragma unroll
    for (int t4 = 0; t4 < NT; t4 += 4) {
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
            if (g < G) {
                const float4 p = *reinterpret_cast<const float4*>(&p_lds[g][t4]);
                const float pw[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[g][0] += pw[e] * __uint_as_float(vr[t4 + e] << 16);
                    acc[g][1] += pw[e] * __uint_as_float(vr[t4 + e] & 0xFFFF0000u);
                }
            }
        }
    }
}

// One workgroup of two wavefronts per (part, KV head, sequence); the r
// residual tokens of a sequence are cut into kResSlots parts of
// ceil(r / kResSlots) <= 64 tokens, and each part into two halves, one per
// wavefront (residual_wave).  The second wavefront hands its maxima, sums and
// weighted values to the first through LDS, which merges them, rotates the
// sum by H so that the merge's inverse rotation H / d returns it (H H = d I;
// not when the values were coded in the caller's basis: the merge then leaves
// the output as it is) and writes one more split-K partial, in slot NC + part.
// A part without tokens writes m = -inf and zeros.
__global__ __launch_bounds__(kResWaves * kWave) void attn_residual_kernel(ResArgs a) {
    __shared__ __align__(16) float p_lds[kResWaves][kMaxGroup][kResWaveTokens];
    __shared__ float2 x_acc[kMaxGroup][kWave];
    __shared__ float x_m[kMaxGroup], x_l[kMaxGroup];
    const int part = blockIdx.x, h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int G = a.G, NC = min(max(a.ws_hdr[1], 1), a.nc_max), rotate = a.ws_hdr[3];
    if ((part | h | b) == 0 && tid == 0) a.ws_hdr[2] = kResSlots;
    const int r = max(0, min(a.res_lens[b], a.r_cap));
    const int ps = (r + kResSlots - 1) / kResSlots;
    const int t0 = part * ps;
    const int n = max(0, min(ps, r - t0));
    const int64_t slot0 = ((int64_t)b * a.Hq + h * G) * (NC + kResSlots) + NC + part;
    if (n == 0) {
        if (wave == 0) {
            for (int g = 0; g < G; ++g) {
                const int64_t slot = slot0 + (int64_t)g * (NC + kResSlots);
                *reinterpret_cast<float2*>(&a.ws_acc[slot * kD + 2 * lane]) = float2{0.f, 0.f};
                if (lane == 0) {
                    a.ws_m[slot] = -INFINITY;
                    a.ws_l[slot] = 0.f;
                }
            }
        }
        return;
    }
    // halves: the first wavefront takes ceil(n / 2) >= 1 tokens, the second the rest
    const int nh = (n + 1) / 2;
    const int nw = wave ? n - nh : nh;
    const int ring0 = max(0, a.seq_lens[b]) % a.r_cap + t0 + (wave ? nh : 0);
    float acc[kMaxGroup][2], mx[kMaxGroup], sm[kMaxGroup];
    if (nw > 16) {
        residual_wave<32>(a, b, h, ring0, nw, lane, p_lds[wave], acc, mx, sm);
    } else if (nw > 0) {
        residual_wave<16>(a, b, h, ring0, nw, lane, p_lds[wave], acc, mx, sm);
    } else {
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
            acc[g][0] = acc[g][1] = 0.f;
            mx[g] = -INFINITY;
            sm[g] = 0.f;
        }
    }
    if (wave == 1) {
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
            if (g < G) {
                x_acc[g][lane] = float2{acc[g][0], acc[g][1]};
                if (lane == 0) {
                    x_m[g] = mx[g];
                    x_l[g] = sm[g];
                }
            }
        }
    }
    __syncthreads();
    if (wave == 1) return;
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) {
        if (g < G) {
            // the first wavefront holds at least one token: M is finite
            const float m1 = x_m[g], M = fmaxf(mx[g], m1);
            const float e0 = exp2f(mx[g] - M), e1 = exp2f(m1 - M);
            const float2 o = x_acc[g][lane];
            float v0 = acc[g][0] * e0 + o.x * e1, v1 = acc[g][1] * e0 + o.y * e1;
            if (rotate) {
                // channels 2 l (v0) and 2 l + 1 (v1): stage h = 1 inside the
                // lane, stages h = 2, 4, ..., 64 between lanes l and l ^ h / 2
                const float w0 = v0 + v1, w1 = v0 - v1;
                v0 = w0;
                v1 = w1;
                hadamard_stage<1>(v0, v1, lane);
                hadamard_stage<2>(v0, v1, lane);
                hadamard_stage<4>(v0, v1, lane);
                hadamard_stage<8>(v0, v1, lane);
                hadamard_stage<16>(v0, v1, lane);
                hadamard_stage<32>(v0, v1, lane);
            }
            const int64_t slot = slot0 + (int64_t)g * (NC + kResSlots);
            *reinterpret_cast<float2*>(&a.ws_acc[slot * kD + 2 * lane]) = float2{v0, v1};
            if (lane == 0) {
                a.ws_m[slot] = M;
                a.ws_l[slot] = sm[g] * e0 + x_l[g] * e1;
            }
        }
    }
}

// ------------------------------------------- merge with the residual window
//
// The residual window and the merge in one launch: a workgroup of eight
// wavefronts per (KV head, sequence).  Wavefront w takes half w % 2 of part
// w / 2 of the window (residual_wave, the same split as attn_residual_kernel)
// and leaves its maxima, sums and weighted values in LDS; after the one
// barrier, wavefront g merges query head g of the group: the chunk partials
// of the compressed tokens (their rows requested at the start, so they arrive
// while the window is computed), rotated back by H / d when the values were
// rotated online, and the eight window partials, which are in the original
// basis already.  The residual slots of the workspace are not used.
constexpr int kMrWaves = kResSlots * kResWaves;   // 8: halves of the window's parts, then query heads
constexpr int kMrBatch = 8;                       // chunk rows per memory round trip

struct MergeResArgs {
    ResArgs r;
    int t_cap;
    float* out;
};

__global__ __launch_bounds__(kMrWaves * kWave) void attn_merge_residual_kernel(MergeResArgs ma) {
    const ResArgs& a = ma.r;
    __shared__ __align__(16) float p_lds[kMrWaves][kMaxGroup][kResWaveTokens];
    __shared__ __align__(16) float r_acc[kMrWaves][kMaxGroup][kD];
    __shared__ float r_m[kMrWaves][kMaxGroup], r_l[kMrWaves][kMaxGroup];
    const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int G = a.G, chunk = max(a.ws_hdr[0], 1), NC = min(max(a.ws_hdr[1], 1), a.nc_max);
    const int rotate = a.ws_hdr[3];

    // ---- the chunk partials of query head h G + wave, requested first
    const int T = max(0, min(a.seq_lens[b], ma.t_cap));
    const int nc = min(NC, (T + chunk - 1) / chunk);
    const int64_t base = ((int64_t)b * a.Hq + h * G + wave) * (NC + kResSlots);
    float m_lane = -INFINITY, l_lane = 0.f, a0[kMrBatch], a1[kMrBatch];
    if (wave < G) {
        if (lane < nc) {
            m_lane = a.ws_m[base + lane];
            l_lane = a.ws_l[base + lane];
        }
#pragma unroll
        for (int u = 0; u < kMrBatch; ++u) {
            const int64_t s = base + min(u, max(nc - 1, 0));
            a0[u] = a.ws_acc[s * kD + lane];
            a1[u] = a.ws_acc[s * kD + lane + 64];
        }
    }

    // ---- the window: half (wave % 2) of part (wave / 2)
    {
        const int part = wave >> 1, half = wave & 1;
        const int r = max(0, min(a.res_lens[b], a.r_cap));
        const int ps = (r + kResSlots - 1) / kResSlots;
        const int t0 = part * ps;
        const int n = max(0, min(ps, r - t0));
        const int nh = (n + 1) / 2;
        const int nw = half ? n - nh : nh;
        const int ring0 = max(0, a.seq_lens[b]) % a.r_cap + t0 + (half ? nh : 0);
        float acc[kMaxGroup][2], mx[kMaxGroup], sm[kMaxGroup];
        if (nw > 16) {
            residual_wave<32>(a, b, h, ring0, nw, lane, p_lds[wave], acc, mx, sm);
        } else if (nw > 0) {
            residual_wave<16>(a, b, h, ring0, nw, lane, p_lds[wave], acc, mx, sm);
        } else {
#pragma unroll
            for (int g = 0; g < kMaxGroup; ++g) {
                acc[g][0] = acc[g][1] = 0.f;
                mx[g] = -INFINITY;
                sm[g] = 0.f;
            }
        }
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
            if (g < G) {
                *reinterpret_cast<float2*>(&r_acc[wave][g][2 * lane]) = float2{acc[g][0], acc[g][1]};
                if (lane == 0) {
                    r_m[wave][g] = mx[g];
                    r_l[wave][g] = sm[g];
                }
            }
        }
    }
    __syncthreads();
    if (wave >= G) return;

    // ---- merge of query head g: lane l holds channels l and l + 64
    const int g = wave;
    float* dst = ma.out + ((int64_t)b * a.Hq + h * G + g) * kD;
    float M = m_lane;
    for (int i = lane + kWave; i < nc; i += kWave) M = fmaxf(M, a.ws_m[base + i]);
    M = wave_max_f32(M);
#pragma unroll
    for (int w = 0; w < kMrWaves; ++w) M = fmaxf(M, r_m[w][g]);
    if (M == -INFINITY) {      // no token at all
        dst[lane] = 0.f;
        dst[lane + 64] = 0.f;
        return;
    }
    const float e_lane = lane < nc ? exp2f(m_lane - M) : 0.f;
    float l = wave_sum_f32(l_lane * e_lane);
    float c0 = 0.f, c1 = 0.f;
    for (int i0 = 0; i0 < nc; i0 += kMrBatch) {
        if (i0) {
#pragma unroll
            for (int u = 0; u < kMrBatch; ++u) {
                const int64_t s = base + min(i0 + u, nc - 1);
                a0[u] = a.ws_acc[s * kD + lane];
                a1[u] = a.ws_acc[s * kD + lane + 64];
            }
        }
#pragma unroll
        for (int u = 0; u < kMrBatch; ++u) {
            const int i = i0 + u;
            if (i < nc) {
                float e;
                if (i < kWave) {
                    e = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(e_lane), i));
                } else {
                    e = exp2f(a.ws_m[base + i] - M);
                    l += a.ws_l[base + i] * e;
                }
                c0 += a0[u] * e;
                c1 += a1[u] * e;
            }
        }
    }
    if (rotate) {              // the chunks' values were rotated: H v / d
        hadamard_lanes(c0, c1, lane);
        const float r0 = (c0 + c1) * (1.0f / kD), r1 = (c0 - c1) * (1.0f / kD);
        c0 = r0;
        c1 = r1;
    }
#pragma unroll
    for (int w = 0; w < kMrWaves; ++w) {
        const float e = exp2f(r_m[w][g] - M);     // 0 for a half without tokens
        l += r_l[w][g] * e;
        c0 += r_acc[w][g][lane] * e;
        c1 += r_acc[w][g][lane + 64] * e;
    }
    dst[lane] = c0 / l;
    dst[lane + 64] = c1 / l;
}

// One new token per sequence into its ring slot; block per sequence.
__global__ __launch_bounds__(kResThreads) void residual_append_kernel(const uint16_t* __restrict__ k_new,
                                                                      const uint16_t* __restrict__ v_new,
                                                                      int Hkv, uint16_t* __restrict__ rk,
                                                                      uint16_t* __restrict__ rv,
                                                                      const int32_t* __restrict__ seq_lens,
                                                                      int32_t* __restrict__ res_lens,
                                                                      int r_cap, uint32_t* status) {
    const int b = blockIdx.x, tid = threadIdx.x;
    const int r = res_lens[b];
    if (r < 0 || r >= r_cap) {
        if (tid == 0 && status) atomicOr(status, DQ_STATUS_WINDOW);
        return;
    }
    const int slot = (max(0, seq_lens[b]) + r) % r_cap;
    for (int i = tid; i < Hkv * kD; i += kResThreads) {
        const int h = i / kD, j = i % kD;
        const int64_t dst = (((int64_t)b * Hkv + h) * r_cap + slot) * kD + j;
        rk[dst] = k_new[(int64_t)b * Hkv * kD + i];
        rv[dst] = v_new[(int64_t)b * Hkv * kD + i];
    }
    __syncthreads();
    if (tid == 0) res_lens[b] = r + 1;
}

// After the oldest n residual tokens were encoded: they become compressed.
__global__ void residual_commit_kernel(int32_t* __restrict__ seq_lens, int32_t* __restrict__ res_lens,
                                       int B, int n, uint32_t* status) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int r = res_lens[b];
    if (r < n) {
        if (status) atomicOr(status, DQ_STATUS_WINDOW);
        return;
    }
    seq_lens[b] += n;
    res_lens[b] = r - n;
}

// Record length in dwords of the instantiation that serves (Ck, Cv); 0 = the
// general kernel.
int compiled_rw(int Ck, int Cv) {
    const int p = (Ck % 4 || Cv % 4) ? 0 : rw_pair(Ck / 4, Cv / 4);
    switch (p) {
        case rw_pair(8, 8): case rw_pair(9, 9): case rw_pair(12, 12): case rw_pair(16, 16):
        case rw_pair(12, 8):
            return p;
        default:
            return 0;
    }
}

// LDS layout for given coding sizes; picks the largest wavefront count that fits.
AttnLayout attn_layout(int pk, int pvb, int Ck, int Cv, int G, bool shared_lut, int rw) {
    const int GP = G <= 4 ? 4 : 8, HG = GP / 4;
    AttnLayout L;
    int off = 0;
    // key table at 0; a distinct value table at a fixed 32 KB (the DS offset field)
    L.lut_k = 0;
    if (shared_lut) {
        L.lut_v = 0;
        off = align16(8 << pk);
    } else {
        L.lut_v = (int)kLutVOffset;
        off = (int)kLutVOffset + align16(8 << pvb);
    }
    L.qlimb = off;
    off += align16((kD / 4) * GP * 16);
    L.qscale = off;
    off += align16(GP * 4);
    L.qsum = off;
    off += align16(GP * 4);
    L.qmu = off;
    off += align16(((kMaxChunk + DQ_MEAN_WINDOW - 1) / DQ_MEAN_WINDOW + 1) * GP * 4);
    L.waves = off;
    int w = 0;
    L.pk = w;                                      // key pairs, then value pairs
    L.pv = w + align16((Ck - kPayloadOffset) * kPairRow);
    L.vtile = w;                                   // reuses the pair arrays
    L.plimb = w + align16(kTile * kVRowT);         // so do the weight digits
    w = std::max(L.pv + align16((Cv - kPayloadOffset) * kPairRow),
                 L.plimb + align16(HG * kTile * 16));
    L.wave_stride = w;
    int nw = (kMaxLds - kPairSlack - off) / w;
    if (nw > max_waves(HG, rw)) nw = max_waves(HG, rw);
    // whole wavefronts per SIMD: tiles go round-robin over the wavefronts, so
    // an uneven split would leave two SIMDs with half again the work
    if (nw > 4) nw &= ~3;
    // the query rotation scratch and the final merge must fit as well
    while (nw > 0 && (nw * w < G * kD * 4 ||
                      off + nw * w < nw * (2 * GP + GP * kD) * 4))
        --nw;
    L.nw = nw;
    L.total = off + nw * w + kPairSlack;
    return L;
}

struct ChunkPlan {
    int chunk, nchunks;
    int64_t slots_max;
};


// Few, large chunks: one workgroup fits per CU (LDS), so the grid is sized to
// about one workgroup per CU (more when the batch has more (sequence, KV head)
// pairs than there are CUs), with chunks of kMinChunkHead..kMaxChunk tokens in
// whole 64-token tiles.  Every workgroup then runs its waves over many tiles
// and the grid ends in whole rounds of the CUs.  At small batches and short
// contexts the lower bound sets the grid: a 256-token chunk is four tiles,
// whose keys and values eight wavefronts decode apart (two per SIMD);
// smaller chunks would double the partials the merge reads for no shorter
// chain.
ChunkPlan chunk_plan(int B, int Hq, int Hkv, int t_cap, int num_cus) {
    ChunkPlan p;
    const int64_t pairs = (int64_t)B * Hkv;
    int64_t nc = std::max<int64_t>((t_cap + kMaxChunk - 1) / kMaxChunk, (num_cus + pairs - 1) / pairs);
    int chunk = (int)((t_cap + nc - 1) / nc);
    chunk = ((chunk + kTile - 1) / kTile) * kTile;
    chunk = std::max(chunk, kMinChunkHead);
    chunk = std::min(chunk, kMaxChunk);
    p.chunk = chunk;
    p.nchunks = (t_cap + chunk - 1) / chunk;
    p.slots_max = ws_slots(B, Hq, t_cap);
    return p;
}


}  // namespace

int launch_decode_symbols(const dq_tables* tab, const uint8_t* records, int64_t n_streams,
                          uint8_t* sym, uint16_t* header, uint32_t* status, hipStream_t stream) {
    TabArgs ta = tab_args(tab);
    const int threads = 256;
    const int64_t blocks = (n_streams + threads - 1) / threads;
    if (blocks > 0x7FFFFFFF) return DQ_ERR_INVALID_ARG;
    decode_symbols_kernel<<<dim3((unsigned)blocks), threads, 0, stream>>>(ta, records, n_streams,
                                                                         sym, header, status);
    return hip_check("decode_symbols launch", hipGetLastError());
}

size_t attention_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap, int32_t d) {
    (void)Hkv;
    const int64_t slots = ws_slots(B, Hq, t_cap);
    return (size_t)kWsHeader + (size_t)(slots * d + 2 * slots) * sizeof(float);
}

bool attention_supports(const dq_tables* tk, const dq_tables* tv) {
    for (const dq_tables* t : {tk, tv}) {
        const int C = t->cfg.record_bytes;
        if (C % 4 || C < 12 || C > 4 * kMaxRecDwords) return false;
    }
    return true;
}

template <int HG, uint32_t LUTV, int RWP, bool FIXED, int WMAX, bool SPLIT = false>
static int launch_w(AttnArgs& a, dim3 grid, hipStream_t stream) {
    if (a.L.nw > WMAX) return DQ_ERR_INVALID_ARG;
    if (SPLIT && 2 * ((a.chunk + kTile - 1) / kTile) > a.L.nw) return DQ_ERR_INVALID_ARG;
    if (int rc = hip_check("hipFuncSetAttribute",
                           hipFuncSetAttribute(
                               reinterpret_cast<const void*>(&attn_partial_kernel<HG, LUTV, RWP, FIXED, WMAX, SPLIT>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, a.L.total)))
        return rc;
    attn_partial_kernel<HG, LUTV, RWP, FIXED, WMAX, SPLIT><<<grid, a.L.nw * kWave, a.L.total, stream>>>(a);
    return hip_check("attn_partial launch", hipGetLastError());
}

// Eight query heads per KV head with at most 8 wavefronts (LDS-bound): the
// 8-wavefront instantiation, which prefetches records.
template <int HG, uint32_t LUTV, int RWP, bool FIXED = false>
static int launch_rw(AttnArgs& a, dim3 grid, hipStream_t stream) {
    constexpr int W = max_waves(HG, RWP);
    // chunks of at most nw / 2 tiles (small batches, short contexts): keys and
    // values in different wavefronts (one shared table, equal record lengths)
    if constexpr (HG == 1 && LUTV == 0 && !FIXED && RWP != 0 && (RWP >> 8) == (RWP & 0xFF))
        if (2 * ((a.chunk + kTile - 1) / kTile) <= a.L.nw) return launch_w<HG, LUTV, RWP, FIXED, W, true>(a, grid, stream);
    if constexpr (HG == 2 && W > 8)
        if (a.L.nw <= 8) return launch_w<HG, LUTV, RWP, FIXED, 8>(a, grid, stream);
    return launch_w<HG, LUTV, RWP, FIXED, W>(a, grid, stream);
}

// Record lengths of the 2.0 / 2.25 / 3.0 / 4.0 bits-per-element budgets at
// head_dim 128 (equal for keys and values, or 3.0 / 2.0) get their own
// instantiation; other lengths take the general one.
template <int HG, uint32_t LUTV>
static int launch_hg(AttnArgs& a, dim3 grid, hipStream_t stream) {
    switch (compiled_rw(a.tk.C, a.tv.C)) {
        case rw_pair(8, 8): return launch_rw<HG, LUTV, rw_pair(8, 8)>(a, grid, stream);
        case rw_pair(9, 9): return launch_rw<HG, LUTV, rw_pair(9, 9)>(a, grid, stream);
        case rw_pair(12, 12): return launch_rw<HG, LUTV, rw_pair(12, 12)>(a, grid, stream);
        case rw_pair(16, 16): return launch_rw<HG, LUTV, rw_pair(16, 16)>(a, grid, stream);
        case rw_pair(12, 8): return launch_rw<HG, LUTV, rw_pair(12, 8)>(a, grid, stream);
        default: return launch_rw<HG, LUTV, 0>(a, grid, stream);
    }
}

int launch_attention_partial(const dq_tables* tk, const dq_tables* tv, const Pages& pg, const uint16_t* q,
                             int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* krec,
                             const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                             const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                             uint32_t* status, hipStream_t stream, int64_t ws_slots_used) {
    if (!attention_supports(tk, tv)) return DQ_ERR_INVALID_ARG;
    const int G = Hq / Hkv;
    AttnArgs a;
    a.tk = tab_args(tk);
    a.tv = tab_args(tv);
    a.shared_lut = (tk == tv || (tk->cfg.levels == tv->cfg.levels &&
                                 tk->cfg.precision_bits == tv->cfg.precision_bits &&
                                 tk->cfg.alpha == tv->cfg.alpha && tk->cfg.head_dim == tv->cfg.head_dim))
                       ? 1 : 0;
    a.L = attn_layout(a.tk.p, a.tv.p, a.tk.C, a.tv.C, G, a.shared_lut != 0, compiled_rw(a.tk.C, a.tv.C));
    if (a.L.nw < 1) return DQ_ERR_INVALID_ARG;
    const ChunkPlan plan = chunk_plan(B, Hq, Hkv, t_cap, cu_count());
    a.q = q;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = G;
    a.t_cap = t_cap;
    a.chunk = plan.chunk;
    a.nchunks = plan.nchunks;
    a.krec = krec;
    a.kmq = kmq;
    a.kms = kms;
    a.vrec = vrec;
    a.seq_lens = seq_lens;
    a.rot_q = tk->cfg.prerotated ? 0 : 1;
    a.rot_out = tv->cfg.prerotated ? 0 : 1;
    // the rotated query and key meet with a factor d (H H = d I)
    a.scale_log2 = scale * 1.4426950408889634f / (a.rot_q ? (float)kD : 1.0f);
    const int64_t slots = ws_slots_used > 0 ? ws_slots_used : plan.slots_max;
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + slots * kD;
    a.ws_l = a.ws_m + slots;
    a.status = status;
    a.pg = pg;
    dim3 grid(a.nchunks, Hkv, B);
    if (a.shared_lut) return G <= 4 ? launch_hg<1, 0>(a, grid, stream) : launch_hg<2, 0>(a, grid, stream);
    return G <= 4 ? launch_hg<1, kLutVOffset>(a, grid, stream) : launch_hg<2, kLutVOffset>(a, grid, stream);
}

int launch_attention_fixed_partial(const Pages& pg, const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                   const uint8_t* krec, const int8_t* kmq, const uint16_t* kms,
                                   const uint8_t* vrec, const int32_t* seq_lens, int32_t t_cap, float scale,
                                   void* ws, uint32_t* status, hipStream_t stream) {
    const int G = Hq / Hkv;
    if (G > 4) return DQ_ERR_INVALID_ARG;
    AttnArgs a{};
    // no tables: the layout keeps a minimal (unused) table region
    a.tk.n = a.tv.n = kD;
    a.tk.M = a.tv.M = 4;
    a.tk.p = a.tv.p = 8;
    a.tk.C = a.tv.C = kFixedRecordBytes;
    a.shared_lut = 1;
    a.L = attn_layout(8, 8, kFixedRecordBytes, kFixedRecordBytes, G, true, rw_pair(9, 9));
    if (a.L.nw < 1) return DQ_ERR_INVALID_ARG;
    const ChunkPlan plan = chunk_plan(B, Hq, Hkv, t_cap, cu_count());
    a.q = q;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = G;
    a.t_cap = t_cap;
    a.chunk = plan.chunk;
    a.nchunks = plan.nchunks;
    a.krec = krec;
    a.kmq = kmq;
    a.kms = kms;
    a.vrec = vrec;
    a.seq_lens = seq_lens;
    a.rot_q = a.rot_out = 1;
    a.scale_log2 = scale * 1.4426950408889634f / (float)kD;
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + plan.slots_max * kD;
    a.ws_l = a.ws_m + plan.slots_max;
    a.status = status;
    a.pg = pg;
    dim3 grid(a.nchunks, Hkv, B);
    return launch_rw<1, 0, rw_pair(9, 9), true>(a, grid, stream);
}

int launch_attention_merge(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* seq_lens,
                           int32_t t_cap, const void* ws, float* out, hipStream_t stream, int64_t ws_slots_used) {
    (void)Hkv;
    const int64_t slots = ws_slots_used > 0 ? ws_slots_used : ws_slots(B, Hq, t_cap);
    const int32_t* hdr = static_cast<const int32_t*>(ws);
    const float* acc = reinterpret_cast<const float*>(static_cast<const uint8_t*>(ws) + kWsHeader);
    const float* m = acc + slots * kD;
    const float* l = m + slots;
    const int nc_max = (int)(slots / ((int64_t)B * Hq)) - kResSlots;
    attn_merge_kernel<<<dim3(Hq, B), kWave, 0, stream>>>(hdr, m, l, acc, seq_lens, Hq, t_cap, nc_max, out);
    return hip_check("attn_merge launch", hipGetLastError());
}

int launch_attention_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                              const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                              const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                              void* ws, hipStream_t stream) {
    const int64_t slots = ws_slots(B, Hq, t_cap);
    ResArgs a;
    a.q = q;
    a.rk = res_k;
    a.rv = res_v;
    a.seq_lens = seq_lens;
    a.res_lens = res_lens;
    a.r_cap = r_cap;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = Hq / Hkv;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.nc_max = (int)(slots / ((int64_t)B * Hq)) - kResSlots;
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + slots * kD;
    a.ws_l = a.ws_m + slots;
    attn_residual_kernel<<<dim3(kResSlots, Hkv, B), kResWaves * kWave, 0, stream>>>(a);
    return hip_check("attn_residual launch", hipGetLastError());
}

int launch_attention_merge_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                    const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                                    const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                                    void* ws, float* out, hipStream_t stream) {
    const int64_t slots = ws_slots(B, Hq, t_cap);
    MergeResArgs m;
    ResArgs& a = m.r;
    a.q = q;
    a.rk = res_k;
    a.rv = res_v;
    a.seq_lens = seq_lens;
    a.res_lens = res_lens;
    a.r_cap = r_cap;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = Hq / Hkv;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.nc_max = (int)(slots / ((int64_t)B * Hq)) - kResSlots;
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + slots * kD;
    a.ws_l = a.ws_m + slots;
    m.t_cap = t_cap;
    m.out = out;
    attn_merge_residual_kernel<<<dim3(Hkv, B), kMrWaves * kWave, 0, stream>>>(m);
    return hip_check("attn_merge_residual launch", hipGetLastError());
}

int launch_residual_append(const uint16_t* k_new, const uint16_t* v_new, int32_t B, int32_t Hkv,
                           uint16_t* res_k, uint16_t* res_v, const int32_t* seq_lens, int32_t* res_lens,
                           int32_t r_cap, uint32_t* status, hipStream_t stream) {
    residual_append_kernel<<<B, kResThreads, 0, stream>>>(k_new, v_new, Hkv, res_k, res_v, seq_lens, res_lens,
                                                          r_cap, status);
    return hip_check("residual_append launch", hipGetLastError());
}

int launch_residual_commit(int32_t* seq_lens, int32_t* res_lens, int32_t B, int32_t n, uint32_t* status,
                           hipStream_t stream) {
    residual_commit_kernel<<<(B + 255) / 256, 256, 0, stream>>>(seq_lens, res_lens, B, n, status);
    return hip_check("residual_commit launch", hipGetLastError());
}

int64_t attention_plan_slots(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap) {
    const ChunkPlan plan = chunk_plan(B, Hq, Hkv, t_cap, cu_count());
    return (int64_t)B * Hq * (plan.nchunks + kResSlots);
}

// ------------------------------------------------ allocation-free workspace
//
// dq_decode_attention_no_alloc keeps its split-K workspace in this array
// instead of caller memory.  Each device that loads the library holds its own
// copy until the process ends; host code reaches it only through the device
// address hipGetSymbolAddress returns (the name itself is a host-side
// stand-in).  Nothing in it has to start at zero: the partial kernel writes
// the header and every slot the merge reads.
static __device__ __align__(256) uint8_t scratch[DQ_NO_ALLOC_SCRATCH_BYTES];

int no_alloc_scratch(void** out) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    if (int rc = hip_check("hipGetDevice", hipGetDevice(&dev))) return rc;
    if (dev < 0 || dev >= kMaxDevices) return DQ_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        if (int rc = hip_check("hipGetSymbolAddress(scratch)", hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))))
            return rc;
        if (!p) return hip_fail("hipGetSymbolAddress(scratch)", hipErrorInvalidSymbol);
        addr[dev] = p;
    }
    *out = addr[dev];
    return DQ_OK;
}

int cu_count() {
    static int cached[kMaxDevices] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    if (cached[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

}  // namespace dq
