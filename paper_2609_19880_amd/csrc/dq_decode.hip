// Decode side: rANS decoding of the fixed-size records (Alg. 2) and decode
// attention over them (Sec. 4.5 "Decoding", App. A Eq. fold-key/fold-value).
//
// decode_attention is split-K over context chunks:
//  * attn_partial: one workgroup per (chunk, KV head, sequence), four
//    wavefronts.  The workgroup stages both rANS lookup tables in LDS and
//    rotates the G query heads that share the KV head (one FWHT in LDS).  Each
//    wavefront then takes 64-token tiles: the tile's 64 K and 64 V records are
//    copied to LDS with 16-byte coalesced loads (fixed stride: the address of a
//    record follows from its token index), and every lane decodes one token's
//    stream.  Keys: the decoded level feeds sum_j q_j m_j directly and the
//    affine terms are applied once per token (Eq. fold-key).  Values: levels go
//    to a 64 x 32 byte tile in LDS, the softmax weight is folded with the
//    token's scale (Eq. fold-value) and each lane accumulates one output channel.
//    Online softmax state stays per wavefront; the four wavefronts are merged
//    in LDS at the end.
//  * attn_merge: log-sum-exp merge of the chunk partials per (sequence, query
//    head), then the inverse rotation of the value basis and the 1/d scale.
#include <math.h>

#include "dq_common.h"

namespace dq {
namespace {

constexpr int kD = 128;         // head_dim of the attention kernels
constexpr int kTile = 64;       // tokens per wavefront tile
constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kVSlice = 32;     // value channels decoded between two PV passes
constexpr int kTargetGroups = 2048;

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

struct AttnLayout {
    int lutk, lutv, qr, qsum, qmu, waves, wave_stride;
    int krec, vrec, vt, pv;   // offsets inside a wave region
    int total;
};

__host__ __device__ inline int align16(int v) { return (v + 15) & ~15; }

__host__ __device__ inline AttnLayout attn_layout(int pk, int pv_bits, int Ck, int Cv, int G,
                                                  int chunk) {
    AttnLayout L;
    int off = 0;
    L.lutk = off;
    off += align16(4 << pk);
    L.lutv = off;
    off += align16(4 << pv_bits);
    // the merge at the end reuses [0, ...) : make it large enough
    const int merge = kAttnWaves * (2 * G + G * kD) * 4;
    if (off < merge) off = align16(merge);
    L.qr = off;
    off += align16(kD * G * 4);
    L.qsum = off;
    off += align16(G * 4);
    L.qmu = off;
    off += align16((chunk / DQ_MEAN_WINDOW) * G * 4);
    L.waves = off;
    int w = 0;
    L.krec = w;
    w += align16(kTile * Ck);
    L.vrec = w;
    w += align16(kTile * Cv);
    L.vt = w;
    w += align16(kTile * kVSlice);
    L.pv = w;
    w += align16(kTile * G * 4);
    // the query rotation before the main loop uses the wave regions as scratch
    if (w * kAttnWaves < G * kD * 4) w = align16((G * kD * 4 + kAttnWaves - 1) / kAttnWaves);
    L.wave_stride = w;
    off += kAttnWaves * w;
    L.total = off;
    return L;
}

struct AttnArgs {
    TabArgs tk, tv;
    const uint16_t* q;
    int Hq, Hkv, t_cap, chunk, nchunks;
    const uint8_t* krec;
    const int8_t* kmq;
    const uint16_t* kms;
    const uint8_t* vrec;
    const int32_t* seq_lens;
    float scale_log2;            // softmax_scale * log2(e) / d
    float* ws_m;                 // [B][Hq][NC]
    float* ws_l;                 // [B][Hq][NC]
    float* ws_acc;               // [B][Hq][NC][d]
    uint32_t* status;
    AttnLayout L;
};

__device__ __forceinline__ uint32_t rd_u32(const uint8_t* p) {
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

__device__ __forceinline__ float rd_half(const uint8_t* p) {
    return half_bits_to_f32((uint16_t)(p[0] | (p[1] << 8)));
}

// One step of Alg. 2 on an LDS-resident record: table lookup, state update
// and up to two renormalization bytes (x >= 2^23 and p <= 12 need no more).
__device__ __forceinline__ uint32_t rans_step(uint32_t& x, int& ptr, const uint32_t* lut,
                                              uint32_t mask, int p, const uint8_t* rb, int C) {
    const uint32_t e = lut[x & mask];
    x = ((e >> 12) & 0xFFFu) * (x >> p) + (e & 0xFFFu);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const bool need = x < kRansL;
        const uint32_t byte = rb[min(ptr, C - 1)];
        x = need ? ((x << 8) | byte) : x;
        ptr += need ? 1 : 0;
    }
    return e >> 24;
}

template <int G>
__global__ __launch_bounds__(kAttnThreads) void attn_partial_kernel(AttnArgs a) {
    extern __shared__ __align__(16) uint8_t smem[];
    const AttnLayout& L = a.L;
    uint32_t* lutk = reinterpret_cast<uint32_t*>(smem + L.lutk);
    uint32_t* lutv = reinterpret_cast<uint32_t*>(smem + L.lutv);
    float* qr = reinterpret_cast<float*>(smem + L.qr);        // [d][G]
    float* qsum = reinterpret_cast<float*>(smem + L.qsum);    // [G]
    float* qmu = reinterpret_cast<float*>(smem + L.qmu);      // [chunk/128][G]

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int T = min(a.seq_lens[b], a.t_cap);
    const int start = c * a.chunk;
    if (start >= T) return;   // the merge ignores chunks past the length

    const int Ck = a.tk.C, Cv = a.tv.C;
    const int pk = a.tk.p, pvb = a.tv.p;
    for (int i = tid; i < (1 << pk); i += kAttnThreads) lutk[i] = a.tk.t.lut[i];
    for (int i = tid; i < (1 << pvb); i += kAttnThreads) lutv[i] = a.tv.t.lut[i];

    // Rotate the G query heads: unnormalized FWHT in fp32 (scratch in the wave regions).
    float* qt = reinterpret_cast<float*>(smem + L.waves);     // [G][d]
    const int hq0 = h * G;
    for (int i = tid; i < G * kD; i += kAttnThreads)
        qt[i] = bf16_to_f32(a.q[((int64_t)b * a.Hq + hq0) * kD + i]);
    __syncthreads();
    for (int hh = 1; hh < kD; hh <<= 1) {
        for (int i = tid; i < G * (kD / 2); i += kAttnThreads) {
            const int g = i / (kD / 2), r = i % (kD / 2);
            const int lo = (r / hh) * 2 * hh + (r % hh);
            const float x0 = qt[g * kD + lo], x1 = qt[g * kD + lo + hh];
            qt[g * kD + lo] = x0 + x1;
            qt[g * kD + lo + hh] = x0 - x1;
        }
        __syncthreads();
    }
    for (int i = tid; i < G * kD; i += kAttnThreads) {
        const int g = i / kD, j = i % kD;
        qr[j * G + g] = qt[i];
    }
    __syncthreads();
    if (tid < G) {
        float s = 0.f;
        for (int j = 0; j < kD; ++j) s += qr[j * G + tid];
        qsum[tid] = s;
    }
    // q . mu_hat for every key-mean window of the chunk
    const int nwin_total = a.t_cap / DQ_MEAN_WINDOW;
    const int w0 = start / DQ_MEAN_WINDOW;
    const int nwin = a.chunk / DQ_MEAN_WINDOW;
    for (int i = tid; i < nwin * G; i += kAttnThreads) {
        const int wi = i / G, g = i % G;
        float s = 0.f;
        if (w0 + wi < nwin_total) {
            const int64_t widx = (int64_t)(b * a.Hkv + h) * nwin_total + w0 + wi;
            const float sc = half_bits_to_f32(a.kms[widx]);
            const int8_t* mq = a.kmq + widx * kD;
            for (int j = 0; j < kD; ++j) s += qr[j * G + g] * (sc * (float)mq[j]);
        }
        qmu[i] = s;
    }
    __syncthreads();

    uint8_t* wreg = smem + L.waves + wave * L.wave_stride;
    uint8_t* krs = wreg + L.krec;
    uint8_t* vrs = wreg + L.vrec;
    uint8_t* vt = wreg + L.vt;
    float* pvw = reinterpret_cast<float*>(wreg + L.pv);

    float m_run[G], l_part[G], acco[G], accv[kD / kVSlice][G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        m_run[g] = -INFINITY;
        l_part[g] = 0.f;
        acco[g] = 0.f;
#pragma unroll
        for (int s = 0; s < kD / kVSlice; ++s) accv[s][g] = 0.f;
    }
    const uint32_t maskk = (1u << pk) - 1u, maskv = (1u << pvb) - 1u;
    const int64_t bh = (int64_t)b * a.Hkv + h;
    bool corrupt = false;

    const int ntiles = a.chunk / kTile;
    for (int tile = wave; tile < ntiles; tile += kAttnWaves) {
        const int t_base = start + tile * kTile;
        if (t_base >= T) break;
        {
            const uint4* src = reinterpret_cast<const uint4*>(a.krec + (bh * a.t_cap + t_base) * Ck);
            uint4* dst = reinterpret_cast<uint4*>(krs);
            for (int i = lane; i < 4 * Ck; i += kWave) dst[i] = src[i];
            const uint4* srcv = reinterpret_cast<const uint4*>(a.vrec + (bh * a.t_cap + t_base) * Cv);
            uint4* dstv = reinterpret_cast<uint4*>(vrs);
            for (int i = lane; i < 4 * Cv; i += kWave) dstv[i] = srcv[i];
        }
        wave_sync();
        const int t = t_base + lane;
        const bool valid = t < T;

        // keys: Eq. (fold-key)
        const uint8_t* rk = krs + lane * Ck;
        const float sk = rd_half(rk), ok = rd_half(rk + 2);
        uint32_t x = rd_u32(rk + 4);
        int ptr = kPayloadOffset;
        float acc[G];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g] = 0.f;
#pragma unroll 2
        for (int j = 0; j < kD; ++j) {
            const float lv = (float)rans_step(x, ptr, lutk, maskk, pk, rk, Ck);
            const float* qj = qr + j * G;
#pragma unroll
            for (int g = 0; g < G; ++g) acc[g] = fmaf(qj[g], lv, acc[g]);
        }
        corrupt |= valid && (x != kRansL || ptr > Ck);
        const float* qm = qmu + ((t / DQ_MEAN_WINDOW) - w0) * G;
        float score[G];
#pragma unroll
        for (int g = 0; g < G; ++g)
            score[g] = valid ? (sk * acc[g] + ok * qsum[g] + qm[g]) * a.scale_log2 : -INFINITY;

        // online softmax; value scale folded into the weight (Eq. fold-value)
        const uint8_t* rv = vrs + lane * Cv;
        const float sv = rd_half(rv), ov = rd_half(rv + 2);
        uint32_t xv = rd_u32(rv + 4);
        int ptrv = kPayloadOffset;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float tmax = wave_max(score[g]);
            const float mn = fmaxf(m_run[g], tmax);
            const float corr = (m_run[g] == -INFINITY) ? 0.f : exp2f(m_run[g] - mn);
            const float p = valid ? exp2f(score[g] - mn) : 0.f;
            l_part[g] = l_part[g] * corr + p;
            acco[g] = acco[g] * corr + p * ov;
#pragma unroll
            for (int s = 0; s < kD / kVSlice; ++s) accv[s][g] *= corr;
            m_run[g] = mn;
            pvw[lane * G + g] = p * sv;
        }

        // values: decode a slice of channels into LDS, then accumulate it
        const int ch = lane & (kVSlice - 1), half = lane / kVSlice;
#pragma unroll
        for (int s = 0; s < kD / kVSlice; ++s) {
#pragma unroll 2
            for (int jj = 0; jj < kVSlice; ++jj)
                vt[lane * kVSlice + jj] = (uint8_t)rans_step(xv, ptrv, lutv, maskv, pvb, rv, Cv);
            wave_sync();
#pragma unroll 4
            for (int tt = 0; tt < kTile / 2; ++tt) {
                const int tok = half * (kTile / 2) + tt;
                const float lv = (float)vt[tok * kVSlice + ch];
                const float* pw = pvw + tok * G;
#pragma unroll
                for (int g = 0; g < G; ++g) accv[s][g] = fmaf(pw[g], lv, accv[s][g]);
            }
            wave_sync();
        }
        corrupt |= valid && (xv != kRansL || ptrv > Cv);
    }
    if (__any(corrupt) && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_CORRUPT);

    // combine the two token halves, then the four wavefronts
    float l_tot[G], o_tot[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int s = 0; s < kD / kVSlice; ++s) accv[s][g] += __shfl_xor(accv[s][g], 32);
        l_tot[g] = wave_sum_f32(l_part[g]);
        o_tot[g] = wave_sum_f32(acco[g]);
    }
    __syncthreads();   // every wavefront is done with the tables
    float* mw = reinterpret_cast<float*>(smem);               // [waves][G]
    float* lw = mw + kAttnWaves * G;                          // [waves][G]
    float* aw = lw + kAttnWaves * G;                          // [waves][G][d]
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if (lane == 0) {
            mw[wave * G + g] = m_run[g];
            lw[wave * G + g] = l_tot[g];
        }
        if (lane < kVSlice) {
#pragma unroll
            for (int s = 0; s < kD / kVSlice; ++s)
                aw[(wave * G + g) * kD + s * kVSlice + lane] = accv[s][g] + o_tot[g];
        }
    }
    __syncthreads();
    const int NC = a.nchunks;
    for (int i = tid; i < G * kD; i += kAttnThreads) {
        const int g = i / kD, j = i % kD;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, mw[w * G + g]);
        float acc = 0.f, l = 0.f;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) {
            const float mv = mw[w * G + g];
            if (mv == -INFINITY) continue;
            const float e = exp2f(mv - M);
            acc += aw[(w * G + g) * kD + j] * e;
            l += lw[w * G + g] * e;
        }
        const int64_t slot = ((int64_t)b * a.Hq + hq0 + g) * NC + c;
        a.ws_acc[slot * kD + j] = acc;
        if (j == 0) {
            a.ws_m[slot] = M;
            a.ws_l[slot] = l;
        }
    }
}

__global__ __launch_bounds__(kD) void attn_merge_kernel(const float* __restrict__ ws_m,
                                                        const float* __restrict__ ws_l,
                                                        const float* __restrict__ ws_acc,
                                                        const int32_t* __restrict__ seq_lens,
                                                        int Hq, int t_cap, int chunk, int NC,
                                                        float* __restrict__ out) {
    __shared__ float o[kD];
    const int hq = blockIdx.x, b = blockIdx.y, j = threadIdx.x;
    const int T = min(seq_lens[b], t_cap);
    float* dst = out + ((int64_t)b * Hq + hq) * kD;
    if (T <= 0) {
        dst[j] = 0.f;
        return;
    }
    const int nc = (T + chunk - 1) / chunk;
    const int64_t base = ((int64_t)b * Hq + hq) * NC;
    float M = -INFINITY;
    for (int c = 0; c < nc; ++c) M = fmaxf(M, ws_m[base + c]);
    float acc = 0.f, l = 0.f;
    for (int c = 0; c < nc; ++c) {
        const float e = exp2f(ws_m[base + c] - M);
        acc += ws_acc[(base + c) * kD + j] * e;
        l += ws_l[base + c] * e;
    }
    o[j] = acc / l;
    __syncthreads();
    // inverse rotation of the value basis: H v / d
    for (int hh = 1; hh < kD; hh <<= 1) {
        float mine = o[j], other = o[j ^ hh];
        __syncthreads();
        o[j] = (j & hh) ? (other - mine) : (mine + other);
        __syncthreads();
    }
    dst[j] = o[j] * (1.0f / kD);
}

int choose_chunk(int B, int Hkv, int t_cap) {
    const int units = (t_cap + 255) / 256;
    long long k = ((long long)B * Hkv * units) / kTargetGroups;
    if (k < 1) k = 1;
    if (k > 16) k = 16;
    if (k > units) k = units;
    return 256 * (int)k;
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
    return hip_check("kernel launch", hipGetLastError());
}

size_t attention_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap, int32_t d) {
    const int chunk = choose_chunk(B, Hkv, t_cap);
    const int64_t NC = (t_cap + chunk - 1) / chunk;
    const int64_t slots = (int64_t)B * Hq * NC;
    return (size_t)(slots * d + 2 * slots) * sizeof(float) + 256;
}

template <int G>
static int launch_g(AttnArgs& a, dim3 grid, hipStream_t stream) {
    if (int rc = hip_check("hipFuncSetAttribute",
                           hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_partial_kernel<G>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, a.L.total)))
        return rc;
    attn_partial_kernel<G><<<grid, kAttnThreads, a.L.total, stream>>>(a);
    return hip_check("kernel launch", hipGetLastError());
}

struct ChunkPlan {
    int chunk, nchunks;
    int64_t slots;
};

static ChunkPlan chunk_plan(int B, int Hq, int Hkv, int t_cap) {
    ChunkPlan p;
    p.chunk = choose_chunk(B, Hkv, t_cap);
    p.nchunks = (t_cap + p.chunk - 1) / p.chunk;
    p.slots = (int64_t)B * Hq * p.nchunks;
    return p;
}

int launch_attention_partial(const dq_tables* tk, const dq_tables* tv, const uint16_t* q,
                             int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* krec,
                             const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                             const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                             uint32_t* status, hipStream_t stream) {
    const int G = Hq / Hkv;
    const ChunkPlan plan = chunk_plan(B, Hq, Hkv, t_cap);
    AttnArgs a;
    a.tk = tab_args(tk);
    a.tv = tab_args(tv);
    a.q = q;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.t_cap = t_cap;
    a.chunk = plan.chunk;
    a.nchunks = plan.nchunks;
    a.krec = krec;
    a.kmq = kmq;
    a.kms = kms;
    a.vrec = vrec;
    a.seq_lens = seq_lens;
    a.scale_log2 = scale * 1.4426950408889634f / (float)kD;
    a.ws_acc = static_cast<float*>(ws);
    a.ws_m = a.ws_acc + plan.slots * kD;
    a.ws_l = a.ws_m + plan.slots;
    a.status = status;
    a.L = attn_layout(a.tk.p, a.tv.p, a.tk.C, a.tv.C, G, a.chunk);
    if (a.L.total > 160 * 1024) return DQ_ERR_INVALID_ARG;
    dim3 grid(a.nchunks, Hkv, B);
    switch (G) {
        case 1: return launch_g<1>(a, grid, stream);
        case 2: return launch_g<2>(a, grid, stream);
        case 3: return launch_g<3>(a, grid, stream);
        case 4: return launch_g<4>(a, grid, stream);
        case 5: return launch_g<5>(a, grid, stream);
        case 6: return launch_g<6>(a, grid, stream);
        case 7: return launch_g<7>(a, grid, stream);
        case 8: return launch_g<8>(a, grid, stream);
        default: return DQ_ERR_INVALID_ARG;
    }
}

int launch_attention_merge(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* seq_lens,
                           int32_t t_cap, const void* ws, float* out, hipStream_t stream) {
    const ChunkPlan plan = chunk_plan(B, Hq, Hkv, t_cap);
    const float* acc = static_cast<const float*>(ws);
    const float* m = acc + plan.slots * kD;
    const float* l = m + plan.slots;
    attn_merge_kernel<<<dim3(Hq, B), kD, 0, stream>>>(m, l, acc, seq_lens, Hq, t_cap, plan.chunk,
                                                      plan.nchunks, out);
    return hip_check("attn_merge launch", hipGetLastError());
}

}  // namespace dq
