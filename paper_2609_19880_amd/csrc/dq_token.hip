// Decode attention over per-token streams: one rANS stream of n = 128 H_kv
// values per token spanning every KV head (the paper's default grouping,
// Sec. 4.1 and Sec. 5.1), decoded once and consumed one KV head at a time as
// Sec. 4.5 ("Decoding") describes.
//
// Work split.  One workgroup per (context chunk, sequence); each wavefront
// takes 64-token tiles, one token per lane, and runs the token's key and
// value streams as two interleaved rANS chains (Alg. 2).  After every 128
// steps (one KV head) the head's G query heads get their q . k products
// (Eq. fold-key, on the matrix cores as the levels appear), the online
// softmax update and P . v (Eq. fold-value, on the 16x16x32 matrix cores);
// the chains then continue into the next head with their state.  All query
// heads' accumulators live in the wavefront: per KV head and group of 4
// query-head slots (one group for up to 4 query heads per KV head, two for up
// to 8), lane l holds slot l / 16 of the group for 8 of the 128 channels.
//
// Record bytes.  Records (C bytes in S-byte slots, S a multiple of 16) are
// stored per 64-token tile with 8-byte chunks outermost: chunk c of the tile's
// token l at c * 512 + l * 8 from the tile, so the 64 lanes of a wavefront
// loading the same chunk read 512 contiguous bytes.  They are read in 8-byte
// chunks into a per-lane ring of 8 dwords in LDS, laid out
// [dword row][lane] so that every lane stays in its own bank; a ninth row
// repeats row 0 so that two consecutive dwords are always rows r, r + 1.  A
// decode step reads the two dwords holding its byte position and takes the
// next 16 bits with a funnel shift and a byte permute.  Every 8 steps a lane
// whose ring holds fewer than 20 bytes from its position writes its next
// chunk (held in registers since the previous refill) and loads the one
// after, and does so once more in the rare case that it is still short: 8
// steps read at most 16 bytes, and their two-dword windows reach at most 19
// bytes past the position.  A chunk is written only while the ring is short,
// so the chunk four back that it replaces lies wholly behind the position
// and is never read again.  Ring rows are masked, so a corrupt stream reads
// garbage inside its ring, never outside; it is flagged at the end (state !=
// L or pointer past the record).
#include <math.h>

#include <algorithm>

#include "dq_attn.h"

namespace dq {
namespace {

constexpr int kD = 128;
constexpr int kTile = 64;
constexpr int kVSlice = 64;
constexpr int kVRowT = 80;               // bytes per token row of the value tile (64 channels + pad)
constexpr int kMaxLds = 160 * 1024;
// wavefronts per workgroup at most: 12 with up to 4 query heads per KV head
// (168 VGPRs), 8 with up to 8 (the accumulators of 64 query heads take 128)
__host__ __device__ constexpr int tok_waves(int HG) { return HG == 1 ? 12 : 8; }
constexpr int kTokSplitWaves = 8;          // split tiles: 4 pairs of wavefronts (at most 256 VGPRs)
constexpr int kTokMaxHeads = 8;           // KV heads per stream (n <= 1024)
constexpr int kTokMaxChunk = 2048;        // bounds the per-window q . mu table
constexpr int kRingRow = 4 * kTile;       // bytes per ring row: one dword per lane
constexpr int kRingRows = 8;              // dwords of record bytes per lane
constexpr int kRingBytes = (kRingRows + 1) * kRingRow;   // + the copy of row 0
constexpr int kGroups = kD / 4;           // 4-step groups per head

struct TokLayout {
    int nw;
    int lut_k, lut_v;   // 8-byte tables (the same offset when K and V share one)
    int qlimb;          // [H_kv][32 groups][4 HG slots] x 16 B (three digit words)
    int qscale, qsum;   // float [H_q]
    int qmu;            // float [windows][H_q]
    int waves;          // first wavefront region
    int wave_stride;
    int ring_k, ring_v; // per wavefront
    int vtile;          // [64 tokens][kVRowT]: levels of a 64-channel slice
    int plimb;          // [HG][64 tokens][16]: weight digits, byte 4 slot + digit (digit 3 zero)
    int total;
};

struct TokArgs {
    TabArgs tk, tv;
    const uint16_t* q;
    int Hq, Hkv, G, t_cap, chunk, nchunks;
    const uint8_t* krec;
    const int8_t* kmq;
    const uint16_t* kms;
    const uint8_t* vrec;
    int k_stride, v_stride;       // bytes per token record (multiples of 16)
    Pages pg;                     // block table of a paged cache (bt null: contiguous)
    const int32_t* seq_lens;
    float scale_log2;             // softmax_scale * log2(e) / d (/ 1 for prerotated keys)
    int rot_q, rot_out;           // keys / values rotated online (tables not prerotated)
    int32_t* ws_hdr;
    float* ws_m;
    float* ws_l;
    float* ws_acc;
    uint32_t* status;
    TokLayout L;
};

// Two steps of Alg. 2 on one ring read, state X = 8 x as in the per-head
// kernel; pb is the lane's bit position in its record (8 x byte position).
//   dwords j = pb >> 5 and j + 1 come from ring rows j mod 8 and the next
//   w = bytes pos .. pos + 3, little-endian = (hi:lo) >> (pb mod 32)
//   r = b_pos << 24 | b_pos+1 << 16 | b_pos+2 << 8 | b_pos+3 (byte reverse)
// r >> (29 - sh) puts the sh bits to shift in at bits 3 and up; what lands in
// the low three bits of X is never read.  Each step reads at most 2 bytes, so
// the second step's bytes are r << sh of the first.
//
// The two steps are split so that the key and value chains of a lane
// overlap: tissue_a requests the ring dwords and the first table word,
// tfinish_a completes the first step, tissue_b requests the second table
// word, tfinish_b completes the second step.  The compiler does not see the
// requested loads, so nothing may read their results until a twait<N> has run
// on them: it waits until at most N LDS or scalar-memory operations are
// outstanding (LDS returns in order; N counts the LDS reads issued after the
// awaited one, and operations the compiler adds in between only make the wait
// stricter).  The finish steps return the table words (levels in their top
// bytes).
struct TChain {
    uint32_t X, pb, w;
    uint64_t rr, e;      // pending: ring dwords (lo, hi), table word
};

template <uint32_t LUT_OFF>
__device__ __forceinline__ void tissue_a(TChain& c, uint32_t ring_lane, uint32_t mask8) {
    uint32_t addr;
    asm("v_lshl_add_u32 %0, %1, 8, %2" : "=v"(addr) : "v"(__builtin_amdgcn_ubfe(c.pb, 5, 3)), "v"(ring_lane));
    asm volatile("ds_read2st64_b32 %0, %2 offset1:1\n\t"
                 "ds_read_b64 %1, %3 offset:%4"
                 : "=&v"(c.rr), "=&v"(c.e)
                 : "v"(addr), "v"(c.X & mask8), "i"(LUT_OFF));
}

template <uint32_t LUT_OFF>
__device__ __forceinline__ void tissue_b(TChain& c, uint32_t mask8) {
    asm volatile("ds_read_b64 %0, %1 offset:%2" : "=&v"(c.e) : "v"(c.X & mask8), "i"(LUT_OFF));
}

template <int N>
__device__ __forceinline__ void twait_a(TChain& c) {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(c.rr), "+v"(c.e) : "i"(N));
}

template <int N>
__device__ __forceinline__ void twait_b(TChain& c) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(c.e) : "i"(N));
}

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// The query digits of one group (16 bytes at LDS address a + off, off a
// constant once unrolled), requested under the same rule: pending until a
// twait_bq that follows it has run.
__device__ __forceinline__ void qissue(uint32_t a, int off, v4u& q) {
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=&v"(q) : "v"(a), "i"(off));
}

template <int N, int HG>
__device__ __forceinline__ void twait_bq(TChain& c, v4u (&q)[HG]) {
    if constexpr (HG == 1)
        asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(c.e), "+v"(q[0]) : "i"(N));
    else
        asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(c.e), "+v"(q[0]), "+v"(q[1]) : "i"(N));
}

// sh of the first step, kept for the second
__device__ __forceinline__ uint32_t tfinish_a(TChain& c, int p3, uint32_t& sh) {
    const uint32_t lo = (uint32_t)c.rr, hi = (uint32_t)(c.rr >> 32);
    const uint32_t w = __builtin_amdgcn_perm(0u, __builtin_amdgcn_alignbit(hi, lo, c.pb), 0x00010203u);
    const uint32_t ea = (uint32_t)c.e;
    const uint32_t y = __umul24(ea, c.X >> p3) + (uint32_t)(c.e >> 32);
    sh = (uint32_t)__builtin_clz(y) & 24u;
    const uint32_t q = w >> (sh ^ 29u);
    asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(c.X) : "v"(y), "v"(sh), "v"(q));
    c.w = w << sh;
    return ea;
}

__device__ __forceinline__ uint32_t tfinish_b(TChain& c, int p3, uint32_t sha) {
    const uint32_t eb = (uint32_t)c.e;
    const uint32_t y = __umul24(eb, c.X >> p3) + (uint32_t)(c.e >> 32);
    const uint32_t sh = (uint32_t)__builtin_clz(y) & 24u;
    const uint32_t q = c.w >> (sh ^ 29u);
    asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(c.X) : "v"(y), "v"(sh), "v"(q));
    asm("v_add3_u32 %0, %1, %2, %3" : "=v"(c.pb) : "v"(c.pb), "v"(sha), "v"(sh));
    return eb;
}

// rec: the lane's first chunk (tile + 8 lane); chunks are 512 bytes apart.
__device__ __forceinline__ uint2 load_chunk(const uint8_t* rec, uint32_t c, uint32_t last) {
    return *reinterpret_cast<const uint2*>(rec + 512u * min(c, last));
}

// Chunk c of the record into ring rows 2 (c mod 4), + 1 (and row 8 for c
// mod 4 = 0).
__device__ __forceinline__ void put_chunk(uint32_t ring_lane, uint32_t c, const uint2& v) {
    const uint32_t a = ring_lane + (c & 3u) * 2u * kRingRow;
    *LDS_PTR(uint32_t, a) = v.x;
    *LDS_PTR(uint32_t, a + kRingRow) = v.y;
    if ((c & 3u) == 0) *LDS_PTR(uint32_t, ring_lane + kRingRows * kRingRow) = v.x;
}

// One chunk per ring toward 8 nc >= pos + 20 (the bytes the next 8 steps can
// read).  thr is 8 (8 nc - 20) - 1 in bits, so the test is one compare.  Both
// rings are written before either chunk load is issued: the loads complete in
// order, so the writes wait only for chunks loaded at earlier refills, never
// for the other ring's load of this group.
__device__ __forceinline__ void refill2(uint32_t pbk, uint32_t& nck, uint32_t& thrk, uint2& nk, uint32_t ring_k,
                                        const uint8_t* kr, uint32_t last_k, uint32_t pbv, uint32_t& ncv,
                                        uint32_t& thrv, uint2& nv, uint32_t ring_v, const uint8_t* vr,
                                        uint32_t last_v) {
    const bool rk = pbk > thrk, rv = pbv > thrv;
    if (rk) put_chunk(ring_k, nck, nk);
    if (rv) put_chunk(ring_v, ncv, nv);
    if (rk) {
        ++nck;
        thrk += 64u;
        nk = load_chunk(kr, nck, last_k);
    }
    if (rv) {
        ++ncv;
        thrv += 64u;
        nv = load_chunk(vr, ncv, last_v);
    }
}

// One chunk for one ring (keys and values decoded by separate wavefronts).
__device__ __forceinline__ void refill1(uint32_t pb, uint32_t& nc, uint32_t& thr, uint2& nxt, uint32_t ring,
                                        const uint8_t* rec, uint32_t last) {
    if (pb > thr) {
        put_chunk(ring, nc, nxt);
        ++nc;
        thr += 64u;
        nxt = load_chunk(rec, nc, last);
    }
}

// The query digits alone (a single chain whose next reads stay in flight).
template <int N>
__device__ __forceinline__ void twait_q(v4u& q) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(q) : "i"(N));
}

// The 128 steps of one KV head on a single chain (the wavefront decodes only
// the keys or only the values of its tile): per step pair the ring dwords
// and the first table word, then the second table word, each awaited before
// it is used; the ring is refilled after every block of 8 steps, whose last
// reads come after the refill's writes.  Keys (KEYS): the query digits of
// group g are requested in its last step pair and the q . k products formed
// as the levels appear; values: the packed levels are returned in vlev.
template <uint32_t LUT, bool KEYS>
__device__ __forceinline__ void chain_head(TChain& c, uint32_t ring, uint32_t mask8, int p3, uint32_t& nc,
                                           uint32_t& thr, uint2& nxt, const uint8_t* rec, uint32_t last,
                                           uint32_t q_lane, v4i (&dk)[3], uint32_t (&vlev)[kGroups]) {
    v4u qd;
#pragma unroll
    for (int grp = 0; grp < kGroups; ++grp) {
        if ((grp & 1) == 0) tissue_a<LUT>(c, ring, mask8);
        uint32_t w[4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const bool more = !((grp & 1) && u == 1);
            uint32_t sh;
            twait_a<0>(c);
            w[2 * u] = tfinish_a(c, p3, sh);
            tissue_b<LUT>(c, mask8);
            if (KEYS && u == 1) {
                qissue(q_lane, (grp * 4) * 16, qd);
                twait_b<1>(c);
            } else {
                twait_b<0>(c);
            }
            w[2 * u + 1] = tfinish_b(c, p3, sh);
            if (more) tissue_a<LUT>(c, ring, mask8);
        }
        const uint32_t lev = pack4(w[0], w[1], w[2], w[3]);
        if constexpr (KEYS) {
            // the digits were requested before the next pair's two reads
            if (grp & 1) twait_q<0>(qd);
            else twait_q<2>(qd);
            dk[0] = mfma(qd.x, lev, dk[0]);
            dk[1] = mfma(qd.y, lev, dk[1]);
            dk[2] = mfma(qd.z, lev, dk[2]);
        } else {
            vlev[grp] = lev;
            asm volatile("" : "+v"(vlev[grp]));
        }
        if (grp & 1) {
            refill1(c.pb, nc, thr, nxt, ring, rec, last);
            // a second chunk only where a lane is still short (rare)
            if (__any(c.pb > thr)) refill1(c.pb, nc, thr, nxt, ring, rec, last);
            // the next block's ring reads come after these writes
            asm volatile("" ::: "memory");
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Accumulators of channel block cb of slice s and slot group hg: one vector
// acc[s][hg][cb] over the KV heads, for query-head slot 4 hg + l / 16 and
// channel 64 s + 16 cb + l mod 16 in lane l.  The head loop is not unrolled,
// so the vectors are rotated by one element per head and the current head is
// always element 0.
typedef float v8f __attribute__((ext_vector_type(kTokMaxHeads)));

__device__ __forceinline__ v8f rot1(const v8f& v) { return v8f{v[1], v[2], v[3], v[4], v[5], v[6], v[7], v[0]}; }

__device__ __forceinline__ float lane_get(float v, int i) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}
__device__ __forceinline__ float lane_set(float v, int i, float x, int lane) { return lane == i ? x : v; }

// PAGED: records and key means through the block table; a separate
// instantiation, so that the contiguous kernel carries none of its state.
// HG: groups of 4 query-head slots per KV head (1: G <= 4, 2: G <= 8).
// SPLIT: one tile per pair of wavefronts, keys and values decoded by
// different wavefronts (chunks of at most nw / 2 tiles: small batches).
template <uint32_t LUTV, bool PAGED, int HG, bool SPLIT = false>
__global__ __launch_bounds__((SPLIT ? kTokSplitWaves : tok_waves(HG)) * kWave) void attn_token_kernel(TokArgs a) {
    constexpr int GS = 4 * HG;                 // query-head slots per KV head
    extern __shared__ __align__(16) uint8_t smem[];
    const TokLayout& L = a.L;
    const int G = a.G, Hkv = a.Hkv, Hq = a.Hq;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int nthr = L.nw * kWave;
    const int c = blockIdx.x, b = blockIdx.z;
    if ((c | b) == 0 && tid == 0) {
        a.ws_hdr[0] = a.chunk;
        a.ws_hdr[1] = a.nchunks;
        a.ws_hdr[2] = 0;          // set by the residual kernel when it runs
        a.ws_hdr[3] = a.rot_out;  // the merge rotates the output back
    }
    const int T = min(a.seq_lens[b], a.t_cap);
    const int start = c * a.chunk;
    if (start >= T) return;   // the merge ignores chunks past the length
    bool bad_page = false;    // a block-table entry outside the pool (read as page 0)

    // ---- prologue: tables, rotated queries, their digits, q . mu per window
    {
        const int Pk = 1 << a.tk.p, Pv = 1 << a.tv.p;
        uint2* lk = reinterpret_cast<uint2*>(smem + L.lut_k);
        for (int i = tid; i < Pk; i += nthr) lk[i] = a.tk.t.lut64[i];
        if (LUTV != 0) {
            uint2* lv = reinterpret_cast<uint2*>(smem + LUTV);
            for (int i = tid; i < Pv; i += nthr) lv[i] = a.tv.t.lut64[i];
        }
    }
    float* qt = reinterpret_cast<float*>(smem + L.waves);          // [H_q][d] scratch
    float* qscale = reinterpret_cast<float*>(smem + L.qscale);
    float* qsum = reinterpret_cast<float*>(smem + L.qsum);
    float* qmu = reinterpret_cast<float*>(smem + L.qmu);
    uint8_t* qlimb = smem + L.qlimb;
    rotate_query_heads(a.q + (int64_t)b * Hq * kD, Hq, Hq, wave, L.nw, lane, qt, qscale, qsum, a.rot_q);
    __syncthreads();
    // digits of head slot r of KV head h at ((h * 32 + j / 4) * GS + r) * 16 + j % 4 (+4, +8)
    for (int i = tid; i < Hkv * GS * kD; i += nthr) {
        const int h = i / (GS * kD), r = (i / kD) % GS, j = i % kD;
        const int g = h * G + r;
        int v = 0;
        if (r < G && qscale[g] > 0.f) {
            v = (int)rintf(qt[g * kD + j] / qscale[g]);
            v = max(-4194304, min(4194304, v));
        }
        int d0, d1, d2;
        digits3(v, d0, d1, d2);
        uint8_t* dst = qlimb + ((h * kGroups + j / 4) * GS + r) * 16 + (j % 4);
        dst[0] = (uint8_t)d0;
        dst[4] = (uint8_t)d1;
        dst[8] = (uint8_t)d2;
        dst[12] = 0;
    }
    const int nwin_total = a.t_cap / DQ_MEAN_WINDOW;
    const int w0 = start / DQ_MEAN_WINDOW;
    const int nwin = (a.chunk + DQ_MEAN_WINDOW - 1) / DQ_MEAN_WINDOW + 1;
    // half a wavefront per (window, KV head), two per pass: lane l takes
    // channels 4 (l % 32) .. 4 (l % 32) + 3 and the KV head's G query heads
    {
        const int r = lane >> 5, c4 = 4 * (lane & 31);
        for (int it = 2 * wave + r; it - r < nwin * Hkv; it += 2 * L.nw) {
            const int wi = it / Hkv, hk = it % Hkv;
            float f[4] = {0.f, 0.f, 0.f, 0.f};
            // windows from the sequence's length on are never used: their
            // block-table entries may be unmapped
            if (it < nwin * Hkv && w0 + wi < nwin_total && (w0 + wi) * DQ_MEAN_WINDOW < T) {
                const int64_t widx = PAGED ? window_index(a.pg, Hkv, a.t_cap, b, hk, w0 + wi, bad_page)
                                           : ((int64_t)b * Hkv + hk) * nwin_total + w0 + wi;
                const float sc = half_bits_to_f32(a.kms[widx]);
                const uint32_t mv = *reinterpret_cast<const uint32_t*>(a.kmq + widx * kD + c4);
#pragma unroll
                for (int k = 0; k < 4; ++k) f[k] = sc * (float)(int8_t)((mv >> (8 * k)) & 0xFF);
            }
            for (int q = 0; q < G; ++q) {
                const int g = hk * G + q;
                float s = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) s = s + qt[g * kD + c4 + k] * f[k];
                s = half_sum_f32(s);
                if ((lane & 31) == 31 && it < nwin * Hkv) qmu[wi * Hq + g] = s;
            }
        }
    }
    __syncthreads();

    // ---- per-wavefront state
    uint8_t* wreg = smem + L.waves + wave * L.wave_stride;
    const uint32_t ring_k = (uint32_t)(L.waves + wave * L.wave_stride + L.ring_k) + 4u * lane;
    const uint32_t ring_v = (uint32_t)(L.waves + wave * L.wave_stride + L.ring_v) + 4u * lane;
    uint8_t* vtile = wreg + L.vtile;
    uint8_t* plimb = wreg + L.plimb;
    // P . v: lane l serves slot l / 16 of each group and channel l % 16 of each
    // 16-channel block; its tr8 reads start at token row 8 (l / 16) +
    // (l % 16) / 2 of a 32-token block, byte 8 (l % 2) of the row's block
    const int pslot = lane >> 4;
    const uint32_t trow = (uint32_t)(8 * (lane >> 4) + ((lane & 15) >> 1));
    const uint32_t a_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.plimb) + trow * 16 + 8 * (lane & 1);
    const uint32_t b_lane = (uint32_t)(L.waves + wave * L.wave_stride + L.vtile) + trow * kVRowT + 8 * (lane & 1);
    const int pk3 = a.tk.p + 3, pv3 = a.tv.p + 3;
    const uint32_t mask8k = ((1u << a.tk.p) - 1u) << 3, mask8v = ((1u << a.tv.p) - 1u) << 3;
    const uint32_t last_k = (uint32_t)(a.k_stride / 8 - 1), last_v = (uint32_t)(a.v_stride / 8 - 1);
    const uint32_t endk = 8u * (uint32_t)a.tk.C, endv = 8u * (uint32_t)a.tv.C;

    // running softmax state of query-head slot GS h + r in lane GS h + r
    float m_vec = -INFINITY, l_vec = 0.f, o_vec = 0.f;
    v8f acc[2][HG][4];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int hg = 0; hg < HG; ++hg)
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) acc[s][hg][cb] = v8f{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    bool corrupt = false;
    const int ntiles = (min(a.chunk, T - start) + kTile - 1) / kTile;

    if constexpr (SPLIT) {
        // One tile per pair of wavefronts.  Per KV head the even wavefront
        // decodes the keys alone and forms the scores and the softmax weights
        // (their digits in one of two weight tiles of its region, the slots'
        // corrections and weight scales beside them), while the odd one
        // decodes the values alone; after the head's barrier the odd one forms
        // P . v with its partner's weights, while the even one goes on to the
        // next head (whose weights go to the other tile).  At the end the even
        // wavefront hands its softmax statistics to the odd one, which alone
        // then holds the pair's partial.
        static_assert(HG == 1, "split tiles: up to 4 query heads");
        const int tile = wave >> 1, role = wave & 1;
        const bool has = tile < ntiles;
        const uint32_t kreg = (uint32_t)(L.waves + (wave & ~1) * L.wave_stride);
        // in the key wavefront's value-tile area: weight tile 1, then
        // [2][GS] corrections, [2][GS] weight scales, and the statistics
        float* kx = reinterpret_cast<float*>(smem + kreg + L.vtile + kTile * 16);
        const int t_base = start + tile * kTile;
        const int t = t_base + lane;
        const bool valid = t < T;
        // a tile never straddles a page
        const int64_t row0 = !has ? 0 : PAGED ? token_row(a.pg, a.t_cap, b, t_base, bad_page)
                                              : (int64_t)b * a.t_cap + t_base;
        const uint8_t* rec = role ? a.vrec + row0 * a.v_stride + 8 * lane : a.krec + row0 * a.k_stride + 8 * lane;
        const uint32_t last = role ? last_v : last_k;
        const uint32_t ring = role ? ring_v : ring_k;
        const uint32_t mask8 = role ? mask8v : mask8k;
        const int p3 = role ? pv3 : pk3;
        TChain ch;
        uint32_t nc = 4, thr = 8u * (8u * 4u - 20u) - 1u;
        uint2 nxt{0u, 0u};
        float sk = 0.f, ok = 0.f, sv = 0.f, ov = 0.f;
        if (has) {
            const uint2 c0 = load_chunk(rec, 0, last), c1 = load_chunk(rec, 1, last), c2 = load_chunk(rec, 2, last),
                        c3 = load_chunk(rec, 3, last);
            nxt = load_chunk(rec, 4, last);
            // the key wavefront also needs the value record's scale and offset
            const uint32_t vh = role ? c0.x : load_chunk(a.vrec + row0 * a.v_stride + 8 * lane, 0, last_v).x;
            put_chunk(ring, 0, c0);
            put_chunk(ring, 1, c1);
            put_chunk(ring, 2, c2);
            put_chunk(ring, 3, c3);
            ch.X = c0.y << 3;
            ch.pb = 64;                             // payload starts at byte 8
            sk = half_lo(c0.x);
            ok = half_hi(c0.x);
            sv = half_lo(vh);
            ov = half_hi(vh);
            asm volatile("" ::: "memory");
        }
        const float* qm = qmu + ((t / DQ_MEAN_WINDOW) - w0) * Hq;
        for (int h = 0; h < Hkv; ++h) {
            v4i dk[3] = {v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}};
            uint32_t vlev[kGroups];
            const int buf = h & 1;
            if (has && role == 0) {
                const uint32_t q_lane = (uint32_t)L.qlimb + (uint32_t)(h * kGroups * GS + (lane & 3)) * 16;
                chain_head<0, true>(ch, ring, mask8, p3, nc, thr, nxt, rec, last, q_lane, dk, vlev);
                // scores of the head's query heads and the online softmax
                float score[4], tmax[4], pw[4], smax[4], corr[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const bool live = r < G;
                    const int g = live ? h * G + r : 0;
                    const float dot = combine(dk[0], dk[1], dk[2], r) * qscale[g];
                    score[r] = (valid && live) ? (sk * dot + ok * qsum[g] + qm[g]) * a.scale_log2 : -INFINITY;
                    tmax[r] = score[r];
                }
                wave_max4_f32(tmax);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int slot = h * GS + r;
                    const float m_old = lane_get(m_vec, slot);
                    const float mn = fmaxf(m_old, tmax[r]);
                    corr[r] = (m_old == -INFINITY || mn == -INFINITY) ? (m_old == mn ? 1.f : 0.f)
                                                                     : __builtin_amdgcn_exp2f(m_old - mn);
                    const float p = (score[r] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(score[r] - mn);
                    const float lt = wave_sum_f32(p);
                    const float ot = wave_sum_f32(p * ov);
                    m_vec = lane_set(m_vec, slot, mn, lane);
                    l_vec = lane_set(l_vec, slot, lane_get(l_vec, slot) * corr[r] + lt, lane);
                    o_vec = lane_set(o_vec, slot, lane_get(o_vec, slot) * corr[r] + ot, lane);
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
                }
                uint8_t* wt = smem + kreg + (buf ? L.vtile : L.plimb);
                *reinterpret_cast<uint4*>(wt + lane * 16) = uint4{wd[0], wd[1], wd[2], wd[3]};
                if (lane == 0) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        kx[buf * GS + r] = corr[r];
                        kx[2 * GS + buf * GS + r] = smax[r] * (1.0f / 4194304.0f);
                    }
                }
            } else if (has) {
                chain_head<LUTV, false>(ch, ring, mask8, p3, nc, thr, nxt, rec, last, 0u, dk, vlev);
            }
            __syncthreads();   // the weights of the head are in LDS
            if (has && role == 1) {
                // ---- P . v over two slices of 64 channels, the partner's weights
                const uint32_t a_pair = kreg + (uint32_t)(buf ? L.vtile : L.plimb) + trow * 16 + 8 * (lane & 1);
                uint64_t pa[2];
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) pa[kb] = lds_tr8(a_pair + kb * 32 * 16);
                const float corr_l = pick4(kx + buf * GS, pslot);
                const float scale_l = pick4(kx + 2 * GS + buf * GS, pslot);
#pragma unroll
                for (int sl = 0; sl < 2; ++sl) {
                    if (sl) wave_sync();   // the first slice's value rows are no longer read
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        *reinterpret_cast<uint4*>(vtile + lane * kVRowT + 16 * q) =
                            uint4{vlev[16 * sl + 4 * q], vlev[16 * sl + 4 * q + 1], vlev[16 * sl + 4 * q + 2],
                                  vlev[16 * sl + 4 * q + 3]};
                    wave_sync();
                    uint64_t vb[kVSlice / 16][2];
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) {
                        vb[cb][0] = lds_tr8(b_lane + 16 * cb);
                        vb[cb][1] = lds_tr8(b_lane + 32 * kVRowT + 16 * cb);
                    }
                    v4i dv[kVSlice / 16];
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) dv[cb] = mfma16(pa[0], vb[cb][0], v4i{0, 0, 0, 0});
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) dv[cb] = mfma16(pa[1], vb[cb][1], dv[cb]);
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) {
                        const float pv =
                            ((float)dv[cb][2] * 65536.0f + (float)dv[cb][1] * 256.0f + (float)dv[cb][0]) * scale_l;
                        v8f tv = acc[sl][0][cb];
                        tv[0] = tv[0] * corr_l + pv;
                        acc[sl][0][cb] = rot1(tv);
                    }
                }
                wave_sync();   // the next head rewrites the value rows
            }
        }
        for (int h = Hkv; h < kTokMaxHeads; ++h)
#pragma unroll
            for (int sl = 0; sl < 2; ++sl)
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) acc[sl][0][cb] = rot1(acc[sl][0][cb]);
        // every stream ends at x = L having read no byte past its record
        if (has) corrupt |= valid && ((ch.X >> 3) != kRansL || ch.pb > (role ? endv : endk));
        // the softmax statistics go to the value wavefront
        float* kst = kx + 4 * GS;
        if (has && role == 0) {
            kst[lane] = m_vec;
            kst[kWave + lane] = l_vec;
            kst[2 * kWave + lane] = o_vec;
        }
        __syncthreads();
        if (has && role == 1) {
            m_vec = kst[lane];
            l_vec = kst[kWave + lane];
            o_vec = kst[2 * kWave + lane];
        } else {
            m_vec = -INFINITY;
        }
    }

    for (int tile = SPLIT ? ntiles : wave; tile < ntiles; tile += L.nw) {
        const int t_base = start + tile * kTile;
        const int t = t_base + lane;               // < t_cap: tiles lie inside the capacity
        const bool valid = t < T;
        // a tile never straddles a page
        const int64_t row0 = PAGED ? token_row(a.pg, a.t_cap, b, t_base, bad_page) : (int64_t)b * a.t_cap + t_base;
        const uint8_t* kr = a.krec + row0 * a.k_stride + 8 * lane;
        const uint8_t* vr = a.vrec + row0 * a.v_stride + 8 * lane;
        // chunks 0..3 (bytes 0..31) cover the first 8 steps from byte 8
        const uint2 k0 = load_chunk(kr, 0, last_k), k1 = load_chunk(kr, 1, last_k), k2 = load_chunk(kr, 2, last_k),
                    k3 = load_chunk(kr, 3, last_k);
        const uint2 v0 = load_chunk(vr, 0, last_v), v1 = load_chunk(vr, 1, last_v), v2 = load_chunk(vr, 2, last_v),
                    v3 = load_chunk(vr, 3, last_v);
        uint2 nk = load_chunk(kr, 4, last_k), nv = load_chunk(vr, 4, last_v);
        wave_sync();   // the previous tile is done with the rings
        put_chunk(ring_k, 0, k0);
        put_chunk(ring_k, 1, k1);
        put_chunk(ring_k, 2, k2);
        put_chunk(ring_k, 3, k3);
        put_chunk(ring_v, 0, v0);
        put_chunk(ring_v, 1, v1);
        put_chunk(ring_v, 2, v2);
        put_chunk(ring_v, 3, v3);
        uint32_t nck = 4, ncv = 4;
        uint32_t thrk = 8u * (8u * 4u - 20u) - 1u, thrv = thrk;
        TChain ck, cv;
        ck.X = k0.y << 3;
        cv.X = v0.y << 3;
        ck.pb = cv.pb = 64;                         // payload starts at byte 8
        const float sk = half_lo(k0.x), ok = half_hi(k0.x);
        const float sv = half_lo(v0.x), ov = half_hi(v0.x);
        const float* qm = qmu + ((t / DQ_MEAN_WINDOW) - w0) * Hq;
        // the rings are read back by this lane only: order the reads after
        // the writes (LDS keeps a wavefront's accesses in order)
        asm volatile("" ::: "memory");

        for (int h = 0; h < Hkv; ++h) {
            v4i dk[HG][3];
#pragma unroll
            for (int hg = 0; hg < HG; ++hg) dk[hg][0] = dk[hg][1] = dk[hg][2] = v4i{0, 0, 0, 0};
            uint32_t vlev[kGroups];
            // the digits of group g are requested in its last step pair, so
            // that the wait for the value step covers them too
            const uint32_t q_lane = (uint32_t)L.qlimb + (uint32_t)(h * kGroups * GS + (lane & 3)) * 16;
            v4u qd[HG];
            // steps in blocks of 8 (two groups): the rings are refilled after
            // each block, so the block's last reads are awaited (and the next
            // block's requested) after the refill; inside a block, step pair u
            // of both chains: wait for the key chain's first reads (the value
            // chain's follow: 2), finish, request its second table word; the
            // same for the value chain (the key chain's word follows: 1); then
            // the second steps (1, and 2 or 0 at the block's end)
#pragma unroll
            for (int grp = 0; grp < kGroups; ++grp) {
                if ((grp & 1) == 0) {
                    tissue_a<0>(ck, ring_k, mask8k);
                    tissue_a<LUTV>(cv, ring_v, mask8v);
                }
                uint32_t kw[4], vw[4];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const bool more = !((grp & 1) && u == 1);
                    uint32_t shk, shv;
                    twait_a<2>(ck);
                    kw[2 * u] = tfinish_a(ck, pk3, shk);
                    tissue_b<0>(ck, mask8k);
                    twait_a<1>(cv);
                    vw[2 * u] = tfinish_a(cv, pv3, shv);
                    tissue_b<LUTV>(cv, mask8v);
                    twait_b<1>(ck);
                    kw[2 * u + 1] = tfinish_b(ck, pk3, shk);
                    if (u == 1) {
                        qissue(q_lane, (grp * GS) * 16, qd[0]);
                        if constexpr (HG == 2) qissue(q_lane, (grp * GS + 4) * 16, qd[1]);
                    }
                    if (more) tissue_a<0>(ck, ring_k, mask8k);
                    if (u == 0) twait_b<2>(cv);
                    else if (more) twait_bq<2>(cv, qd);
                    else twait_bq<0>(cv, qd);
                    vw[2 * u + 1] = tfinish_b(cv, pv3, shv);
                    if (more) tissue_a<LUTV>(cv, ring_v, mask8v);
                }
                const uint32_t lk = pack4(kw[0], kw[1], kw[2], kw[3]);
                vlev[grp] = pack4(vw[0], vw[1], vw[2], vw[3]);
                asm volatile("" : "+v"(vlev[grp]));
#pragma unroll
                for (int hg = 0; hg < HG; ++hg) {
                    dk[hg][0] = mfma(qd[hg].x, lk, dk[hg][0]);
                    dk[hg][1] = mfma(qd[hg].y, lk, dk[hg][1]);
                    dk[hg][2] = mfma(qd[hg].z, lk, dk[hg][2]);
                }
                if (grp & 1) {
                    refill2(ck.pb, nck, thrk, nk, ring_k, kr, last_k, cv.pb, ncv, thrv, nv, ring_v, vr, last_v);
                    // a second chunk only where a lane is still short (rare): the
                    // test is one wavefront vote, so blocks where none is skip it
                    if (__any(ck.pb > thrk || cv.pb > thrv))
                        refill2(ck.pb, nck, thrk, nk, ring_k, kr, last_k, cv.pb, ncv, thrv, nv, ring_v, vr, last_v);
                    // the next block's ring reads come after these writes
                    asm volatile("" ::: "memory");
                }
                __builtin_amdgcn_sched_barrier(0);
            }

            // ---- scores of the head's query heads and the online softmax,
            //      at a raised issue priority: its chains of wavefront
            //      reductions then wait less behind the other wavefronts'
            //      decode steps (1.5 % less time at G = 4, 2.3 % at G = 8;
            //      raising the decode instead, as the per-head kernel does,
            //      was 1 % slower here)
            __builtin_amdgcn_s_setprio(1);
            float corr[GS], pscale[GS];
            int pint[GS];
            // four slots at a time, their tile maxima reduced together
#pragma unroll
            for (int hg = 0; hg < HG; ++hg) {
                float score[4], tmax[4], pw[4], smax[4];
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int r = 4 * hg + rr;
                    const bool live = r < G;
                    const int g = live ? h * G + r : 0;       // slots past G take no query head
                    const float dot = combine(dk[hg][0], dk[hg][1], dk[hg][2], rr) * qscale[g];
                    score[rr] = (valid && live) ? (sk * dot + ok * qsum[g] + qm[g]) * a.scale_log2 : -INFINITY;
                    tmax[rr] = score[rr];
                }
                wave_max4_f32(tmax);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int r = 4 * hg + rr;
                    const int slot = h * GS + r;
                    const float m_old = lane_get(m_vec, slot);
                    const float mn = fmaxf(m_old, tmax[rr]);
                    corr[r] = (m_old == -INFINITY || mn == -INFINITY) ? (m_old == mn ? 1.f : 0.f)
                                                                      : __builtin_amdgcn_exp2f(m_old - mn);
                    const float p = (score[rr] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(score[rr] - mn);
                    const float lt = wave_sum_f32(p);
                    const float ot = wave_sum_f32(p * ov);
                    m_vec = lane_set(m_vec, slot, mn, lane);
                    l_vec = lane_set(l_vec, slot, lane_get(l_vec, slot) * corr[r] + lt, lane);
                    o_vec = lane_set(o_vec, slot, lane_get(o_vec, slot) * corr[r] + ot, lane);
                    pw[rr] = p * sv;                          // >= 0: scales are non-negative
                    smax[rr] = pw[rr];
                }
                wave_max4_f32(smax);
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int r = 4 * hg + rr;
                    pscale[r] = smax[rr] * (1.0f / 4194304.0f);
                    const float inv = smax[rr] > 0.f ? 4194304.0f * __builtin_amdgcn_rcpf(smax[rr]) : 0.f;
                    pint[r] = min(4194304, (int)rintf(pw[rr] * inv));
                }
            }
            // weight digits -> LDS, one 16-byte token row per slot group: byte
            // 4 r + d holds digit d of slot r (byte 4 r + 3 stays zero)
            float corr_l[HG], scale_l[HG];
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
                corr_l[hg] = pick4(corr + 4 * hg, pslot);
                scale_l[hg] = pick4(pscale + 4 * hg, pslot);
            }

            __builtin_amdgcn_s_setprio(0);
            // ---- P . v over two slices of 64 channels
            wave_sync();   // the weight rows are read by other lanes
            uint64_t pa[HG][2];
#pragma unroll
            for (int hg = 0; hg < HG; ++hg)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) pa[hg][kb] = lds_tr8(a_lane + hg * (kTile * 16) + kb * 32 * 16);
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                if (sl) wave_sync();   // the first slice's value rows are no longer read
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *reinterpret_cast<uint4*>(vtile + lane * kVRowT + 16 * q) =
                        uint4{vlev[16 * sl + 4 * q], vlev[16 * sl + 4 * q + 1], vlev[16 * sl + 4 * q + 2],
                              vlev[16 * sl + 4 * q + 3]};
                wave_sync();
                // all operands first, then the product chains
                uint64_t vb[kVSlice / 16][2];
#pragma unroll
                for (int cb = 0; cb < kVSlice / 16; ++cb) {
                    vb[cb][0] = lds_tr8(b_lane + 16 * cb);
                    vb[cb][1] = lds_tr8(b_lane + 32 * kVRowT + 16 * cb);
                }
#pragma unroll
                for (int hg = 0; hg < HG; ++hg) {
                    v4i dv[kVSlice / 16];
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) dv[cb] = mfma16(pa[hg][0], vb[cb][0], v4i{0, 0, 0, 0});
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) dv[cb] = mfma16(pa[hg][1], vb[cb][1], dv[cb]);
#pragma unroll
                    for (int cb = 0; cb < kVSlice / 16; ++cb) {
                        const float pv =
                            ((float)dv[cb][2] * 65536.0f + (float)dv[cb][1] * 256.0f + (float)dv[cb][0]) *
                            scale_l[hg];
                        v8f t = acc[sl][hg][cb];
                        t[0] = t[0] * corr_l[hg] + pv;
                        acc[sl][hg][cb] = rot1(t);
                    }
                }
            }
            wave_sync();   // the next head rewrites the weight and value rows
        }
        for (int h = Hkv; h < kTokMaxHeads; ++h)
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int hg = 0; hg < HG; ++hg)
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) acc[s][hg][cb] = rot1(acc[s][hg][cb]);
        // every stream ends at x = L having read no byte past its record
        corrupt |= valid && ((ck.X >> 3) != kRansL || ck.pb > endk);
        corrupt |= valid && ((cv.X >> 3) != kRansL || cv.pb > endv);
    }
    if (__any(corrupt) && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_CORRUPT);
    if (PAGED && __any(bad_page) && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_PAGE);

    // ---- merge the wavefronts of the workgroup, one KV head at a time
    const int NC = a.nchunks;
    float* mw = reinterpret_cast<float*>(smem);        // [nw][GS]
    float* lw = mw + L.nw * GS;                        // [nw][GS]
    float* aw = lw + L.nw * GS;                        // [nw][GS][d]
    for (int h = 0; h < Hkv; ++h) {
        float av[2][HG][4];
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int hg = 0; hg < HG; ++hg)
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    av[s][hg][cb] = acc[s][hg][cb][0];
                    acc[s][hg][cb] = rot1(acc[s][hg][cb]);
                }
        __syncthreads();   // LDS free (first head) / previous head merged
        float ovs[GS];
#pragma unroll
        for (int r = 0; r < GS; ++r) {
            const int slot = h * GS + r;
            const float mv = lane_get(m_vec, slot), lv = lane_get(l_vec, slot);
            ovs[r] = lane_get(o_vec, slot);
            if (lane == 0) {
                mw[wave * GS + r] = mv;
                lw[wave * GS + r] = lv;
            }
        }
#pragma unroll
        for (int hg = 0; hg < HG; ++hg) {
            const float ovt = pick4(ovs + 4 * hg, pslot);
            float* row = aw + (wave * GS + 4 * hg + pslot) * kD + (lane & 15);
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) row[s * kVSlice + cb * 16] = av[s][hg][cb] + ovt;
        }
        __syncthreads();
        for (int i = tid; i < G * kD; i += nthr) {
            const int r = i / kD, j = i % kD;
            float M = -INFINITY;
            for (int w = 0; w < L.nw; ++w) M = fmaxf(M, mw[w * GS + r]);
            float acc_o = 0.f, l = 0.f;
            for (int w = 0; w < L.nw; ++w) {
                const float mv = mw[w * GS + r];
                if (mv == -INFINITY) continue;
                const float e = exp2f(mv - M);
                acc_o += aw[(w * GS + r) * kD + j] * e;
                l += lw[w * GS + r] * e;
            }
            const int64_t slot = ((int64_t)b * Hq + h * G + r) * (NC + kResSlots) + c;
            a.ws_acc[slot * kD + j] = acc_o;
            if (j == 0) {
                a.ws_m[slot] = M;
                a.ws_l[slot] = l;
            }
        }
    }
}

TokLayout tok_layout(int pk, int pv, bool shared_lut, int Hq, int Hkv, int chunk, int nw, int HG) {
    TokLayout L;
    int off = 0;
    L.lut_k = off;
    off += 8 << pk;
    L.lut_v = shared_lut ? L.lut_k : off;
    if (!shared_lut) off += 8 << pv;
    L.qlimb = off;
    off += Hkv * kGroups * 4 * HG * 16;
    L.qscale = off;
    off += 4 * Hq;
    L.qsum = off;
    off += 4 * Hq;
    L.qmu = off;
    off += 4 * Hq * ((chunk + DQ_MEAN_WINDOW - 1) / DQ_MEAN_WINDOW + 1);
    off = (off + 15) & ~15;
    L.waves = off;
    L.ring_k = 0;
    L.ring_v = kRingBytes;
    L.vtile = 2 * kRingBytes;
    L.plimb = L.vtile + kTile * kVRowT;
    L.wave_stride = (L.plimb + HG * kTile * 16 + 15) & ~15;
    L.nw = nw;
    // the prologue's query scratch and the epilogue's merge buffers use the
    // wavefront regions
    const int scratch = std::max(Hq * kD * 4, nw * 4 * HG * (kD + 2) * 4);
    L.total = L.waves + std::max(nw * L.wave_stride, scratch);
    return L;
}

}  // namespace

// At least one workgroup per CU where the batch allows it, chunks of at most
// kTokMaxChunk tokens and at least kMinChunk (two tiles: at batch 1 a
// token's 1024-step chains bound the time, so more, smaller workgroups
// shorten it, one decoding wavefront per SIMD).
int32_t token_chunk(int32_t B, int32_t t_cap) {
    const int64_t nc = std::max<int64_t>((t_cap + kTokMaxChunk - 1) / kTokMaxChunk, (cu_count() + B - 1) / B);
    int chunk = (int)((t_cap + nc - 1) / nc);
    chunk = ((chunk + kTile - 1) / kTile) * kTile;
    chunk = std::max(chunk, kMinChunk);
    return std::min(chunk, kTokMaxChunk);
}

namespace {

template <uint32_t LUTV, int HG>
int launch_token_kernel(const TokArgs& a, dim3 grid, int nw, hipStream_t stream) {
    const bool paged = a.pg.bt != nullptr;
    // chunks of at most 4 tiles (small batches, short contexts): keys and
    // values in different wavefronts (up to 4 query heads, when LDS holds 8
    // wavefronts)
    if constexpr (HG == 1) {
        TokArgs s = a;
        s.L = tok_layout(a.tk.p, a.tv.p, a.L.lut_v == a.L.lut_k, a.Hq, a.Hkv, a.chunk, kTokSplitWaves, 1);
        // (two 4096-entry tables leave no room for 8 wavefronts: both chains in one)
        if (2 * ((a.chunk + kTile - 1) / kTile) <= kTokSplitWaves && s.L.total <= kMaxLds) {
            const void* fn = paged ? reinterpret_cast<const void*>(&attn_token_kernel<LUTV, true, 1, true>)
                                   : reinterpret_cast<const void*>(&attn_token_kernel<LUTV, false, 1, true>);
            if (int rc = hip_check("hipFuncSetAttribute",
                                   hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, s.L.total)))
                return rc;
            if (paged)
                attn_token_kernel<LUTV, true, 1, true><<<grid, kTokSplitWaves * kWave, (size_t)s.L.total, stream>>>(s);
            else
                attn_token_kernel<LUTV, false, 1, true><<<grid, kTokSplitWaves * kWave, (size_t)s.L.total, stream>>>(s);
            return hip_check("attn_token launch", hipGetLastError());
        }
    }
    const void* fn = paged ? reinterpret_cast<const void*>(&attn_token_kernel<LUTV, true, HG>)
                           : reinterpret_cast<const void*>(&attn_token_kernel<LUTV, false, HG>);
    if (int rc = hip_check("hipFuncSetAttribute",
                           hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, a.L.total)))
        return rc;
    const size_t smem = (size_t)a.L.total;
    if (paged)
        attn_token_kernel<LUTV, true, HG><<<grid, nw * kWave, smem, stream>>>(a);
    else
        attn_token_kernel<LUTV, false, HG><<<grid, nw * kWave, smem, stream>>>(a);
    return hip_check("attn_token launch", hipGetLastError());
}

template <int HG>
int launch_token_hg(const TokArgs& a, dim3 grid, int nw, bool shared, hipStream_t stream) {
    switch (shared ? 0u : (uint32_t)a.L.lut_v) {
        case 0: return launch_token_kernel<0, HG>(a, grid, nw, stream);
        case 8u << 8: return launch_token_kernel<8u << 8, HG>(a, grid, nw, stream);
        case 8u << 9: return launch_token_kernel<8u << 9, HG>(a, grid, nw, stream);
        case 8u << 10: return launch_token_kernel<8u << 10, HG>(a, grid, nw, stream);
        case 8u << 11: return launch_token_kernel<8u << 11, HG>(a, grid, nw, stream);
        case 8u << 12: return launch_token_kernel<8u << 12, HG>(a, grid, nw, stream);
        default: return DQ_ERR_INVALID_ARG;
    }
}

}  // namespace

int launch_attention_token_partial(const dq_tables* tk, const dq_tables* tv, const Pages& pg, const uint16_t* q,
                                   int32_t B,
                                   int32_t Hq, int32_t Hkv, const uint8_t* krec, int32_t k_stride,
                                   const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                                   int32_t v_stride, const int32_t* seq_lens, int32_t t_cap, float scale,
                                   void* ws, uint32_t* status, hipStream_t stream) {
    TokArgs a;
    a.tk = tab_args(tk);
    a.tv = tab_args(tv);
    const bool shared = tk == tv;
    a.q = q;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = Hq / Hkv;
    a.t_cap = t_cap;
    a.chunk = token_chunk(B, t_cap);
    a.nchunks = (t_cap + a.chunk - 1) / a.chunk;
    a.krec = krec;
    a.kmq = kmq;
    a.kms = kms;
    a.vrec = vrec;
    a.k_stride = k_stride;
    a.v_stride = v_stride;
    a.pg = pg;
    a.seq_lens = seq_lens;
    a.rot_q = tk->cfg.prerotated ? 0 : 1;
    a.rot_out = tv->cfg.prerotated ? 0 : 1;
    a.scale_log2 = scale * 1.4426950408889634f / (a.rot_q ? (float)kD : 1.0f);
    const int64_t slots = ws_slots(B, Hq, t_cap);
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + slots * kD;
    a.ws_l = a.ws_m + slots;
    a.status = status;
    if (a.G < 1 || a.G > 8) return DQ_ERR_INVALID_ARG;
    const int HG = a.G > 4 ? 2 : 1;
    int nw = tok_waves(HG);
    for (; nw > 0; --nw) {
        a.L = tok_layout(a.tk.p, a.tv.p, shared, Hq, Hkv, a.chunk, nw, HG);
        if (a.L.total <= kMaxLds) break;
    }
    if (nw == 0) return DQ_ERR_INVALID_ARG;
    const dim3 grid(a.nchunks, 1, B);
    return HG == 1 ? launch_token_hg<1>(a, grid, nw, shared, stream) : launch_token_hg<2>(a, grid, nw, shared, stream);
}

}  // namespace dq
