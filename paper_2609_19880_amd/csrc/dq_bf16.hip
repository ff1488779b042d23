// BF16 decode attention over an uncompressed cache: the comparator of the
// compressed path, on the same shapes (K and V bf16 [B][Hkv][t_cap][d] in the
// original basis), writing the same split-K partials so that attn_merge_kernel
// finishes it.  It is the textbook computation the residual window does for a
// few tokens, at full context; a step reads 2 x 256 bytes per (token, KV head)
// instead of the records' 72.  The kernel is a plain flash-decode built to
// stream those bytes at HBM speed, so that the comparison is with a competent
// uncompressed baseline.
//
// One workgroup of 4 wavefronts per (chunk, KV head, sequence); each
// wavefront takes 32-token tiles and requests all of a tile's key and value
// bytes (16 KB) before it waits for any of them.
//   Logits on the matrix cores: S^T (16 tokens x 16 query-head columns) =
//   K (16 x 32 channels) Q^T (32 x 16), v_mfma_f32_16x16x32_bf16, four
//   32-channel blocks.  Lane l loads 16 bytes of key row l mod 16 at channel
//   8 (l / 16) of each block, which is the A operand as it stands; the query
//   (head l mod 16, the same channels) is the B operand, held in registers
//   for the whole chunk.  Products of bf16 values are exact in fp32.
//   Result: lane l holds head l mod 16 for tokens 4 (l / 16) + i, i < 4.
//   Online softmax per head: the four lanes of a head hold 8 of the tile's
//   32 logits each; the tile maximum is reduced over them, the sum is kept
//   per lane and reduced once at the end.
//   Weighted values on the VALU in fp32: lane l takes channels 8 (l mod 16)
//   .. + 7 of tokens 4 i + l / 16, i < 8 (each 16-byte load instruction
//   reads four whole 256-byte rows), for every query head; the weights come
//   from LDS, one 16-byte broadcast read per token and 4 heads.  The four
//   token groups are summed at the end of the chunk.
// The chunk's value sum is rotated (H acc) before it is stored, since the
// merge undoes the rotation of the compressed path (H H = d I).
#include <math.h>

#include <algorithm>

#include "dq_common.h"

namespace dq {
namespace {

constexpr int kD = 128;
constexpr int kTile = 32;                 // tokens per wavefront pass
constexpr int kBlk = kTile / 16;          // 16-token blocks of the logits
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kPass = kWaves * kTile;     // tokens per workgroup pass
constexpr int kMaxChunkB = 16384;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct B16Args {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* seq_lens;
    int Hq, Hkv, G, t_cap, chunk, nchunks;
    float scale_log2;
    int32_t* ws_hdr;
    float* ws_m;
    float* ws_l;
    float* ws_acc;
};

__device__ __forceinline__ f32x4 mfma_bf16(const uint4& a, const uint4& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                    0, 0, 0);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// GP: query-head slots (4 or 8), G <= GP of them live
template <int GP>
__global__ __launch_bounds__(kThreads) void bf16_partial_kernel(B16Args a) {
    __shared__ __align__(16) float pw[kWaves][kTile][GP];     // softmax weights, [token][head]
    __shared__ float wm[kWaves][GP], wl[kWaves][GP];
    __shared__ __align__(16) float wacc[kWaves][GP][kD];
    __shared__ float rot[GP * kD];
    __shared__ float gm[GP], gl[GP];
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int G = a.G, NC = a.nchunks;
    if ((c | h | b) == 0 && tid == 0) {
        a.ws_hdr[0] = a.chunk;
        a.ws_hdr[1] = a.nchunks;
        a.ws_hdr[2] = 0;
        a.ws_hdr[3] = 1;          // partials are stored rotated (H acc)
    }
    const int T = max(0, min(a.seq_lens[b], a.t_cap));
    const int start = c * a.chunk;
    if (start >= T) return;     // the merge ignores chunks past the length
    const int hq0 = h * G;
    const int col = lane & 15, grp = lane >> 4;

    // the query as the B operand: head col, channels 32 kb + 8 grp .. + 7
    // (read as 16-bit values: the query carries no alignment guarantee)
    uint4 qb[kD / 32];
#pragma unroll
    for (int kb = 0; kb < kD / 32; ++kb) {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if (col < G) {
            const uint16_t* qp = a.q + ((int64_t)b * a.Hq + hq0 + col) * kD + 32 * kb + 8 * grp;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = (uint32_t)qp[2 * e] | ((uint32_t)qp[2 * e + 1] << 16);
        }
        qb[kb] = uint4{w[0], w[1], w[2], w[3]};
    }

    const int64_t row0 = ((int64_t)b * a.Hkv + h) * a.t_cap;
    const uint16_t* kbase = a.k + row0 * kD + 8 * grp;           // + token * kD + 32 kb
    const uint16_t* vbase = a.v + row0 * kD + 8 * col;           // + token * kD
    float m_run = -INFINITY, l_run = 0.f;                        // head col (partial sum over this lane)
    float acc[GP][8];
#pragma unroll
    for (int g = 0; g < GP; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;

    const int ntiles = (min(a.chunk, T - start) + kTile - 1) / kTile;
    for (int tile = wave; tile < ntiles; tile += kWaves) {
        const int t_base = start + tile * kTile;   // the tile lies inside the capacity
        // ---- every load of the tile first
        uint4 kr[kBlk][kD / 32], vr[kTile / 4];
#pragma unroll
        for (int blk = 0; blk < kBlk; ++blk)
#pragma unroll
            for (int kb = 0; kb < kD / 32; ++kb)
                kr[blk][kb] = *reinterpret_cast<const uint4*>(kbase + (int64_t)(t_base + 16 * blk + col) * kD + 32 * kb);
#pragma unroll
        for (int i = 0; i < kTile / 4; ++i)
            vr[i] = *reinterpret_cast<const uint4*>(vbase + (int64_t)(t_base + 4 * i + grp) * kD);

        // ---- logits: S^T blocks of 16 tokens
        f32x4 s[kBlk];
#pragma unroll
        for (int blk = 0; blk < kBlk; ++blk) {
            f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < kD / 32; ++kb) d = mfma_bf16(kr[blk][kb], qb[kb], d);
            s[blk] = d;
        }
        // ---- online softmax of head col over the tile's 32 tokens
        float x[4 * kBlk], mt = -INFINITY;
#pragma unroll
        for (int blk = 0; blk < kBlk; ++blk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int t = t_base + 16 * blk + 4 * grp + i;
                x[4 * blk + i] = t < T ? s[blk][i] * a.scale_log2 : -INFINITY;
                mt = fmaxf(mt, x[4 * blk + i]);
            }
        mt = fmaxf(mt, xor_lane<16>(mt, lane));
        mt = fmaxf(mt, xor_lane<32>(mt, lane));
        const float mn = fmaxf(m_run, mt);
        const float corr = mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - mn);
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 4 * kBlk; ++e) {
            // v_exp_f32 directly: arguments are <= 0 and results that would be
            // denormal may flush to zero
            const float p = x[e] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(x[e] - mn);
            psum += p;
            if (col < GP) pw[wave][16 * (e >> 2) + 4 * grp + (e & 3)][col] = p;
        }
        l_run = l_run * corr + psum;
        m_run = mn;
#pragma unroll
        for (int g = 0; g < GP; ++g) {
            const float cg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(corr), g));
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[g][e] *= cg;
        }
        wave_sync();   // the weights are read by other lanes

        // ---- weighted values; the tile's tokens past the length carry zero
        //      weight, and their rows (which may hold anything) are zeroed
        const bool tail = t_base + kTile > T;
#pragma unroll
        for (int i = 0; i < kTile / 4; ++i) {
            const int tl = 4 * i + grp;
            uint4 w = vr[i];
            if (tail && t_base + tl >= T) w = uint4{0u, 0u, 0u, 0u};
            const float v[8] = {bf_lo(w.x), bf_hi(w.x), bf_lo(w.y), bf_hi(w.y),
                                bf_lo(w.z), bf_hi(w.z), bf_lo(w.w), bf_hi(w.w)};
            float p[GP];
#pragma unroll
            for (int g4 = 0; g4 < GP; g4 += 4) {
                const float4 pv = *reinterpret_cast<const float4*>(&pw[wave][tl][g4]);
                p[g4] = pv.x;
                p[g4 + 1] = pv.y;
                p[g4 + 2] = pv.z;
                p[g4 + 3] = pv.w;
            }
#pragma unroll
            for (int g = 0; g < GP; ++g)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[g][e] += p[g] * v[e];
        }
        wave_sync();   // pw is rewritten by the next tile
    }

    // ---- sum the four token groups, then merge the wavefronts
    l_run += xor_lane<16>(l_run, lane);
    l_run += xor_lane<32>(l_run, lane);
#pragma unroll
    for (int g = 0; g < GP; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[g][e] += xor_lane<16>(acc[g][e], lane);
            acc[g][e] += xor_lane<32>(acc[g][e], lane);
        }
    if (lane < GP) {
        wm[wave][lane] = m_run;
        wl[wave][lane] = l_run;
    }
    if (grp == 0) {
#pragma unroll
        for (int g = 0; g < GP; ++g) {
            *reinterpret_cast<float4*>(&wacc[wave][g][8 * col]) = float4{acc[g][0], acc[g][1], acc[g][2], acc[g][3]};
            *reinterpret_cast<float4*>(&wacc[wave][g][8 * col + 4]) =
                float4{acc[g][4], acc[g][5], acc[g][6], acc[g][7]};
        }
    }
    __syncthreads();
    if (tid < GP) {
        float M = -INFINITY, l = 0.f;
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wm[w][tid]);
        for (int w = 0; w < kWaves; ++w)
            if (wm[w][tid] != -INFINITY) l += wl[w][tid] * exp2f(wm[w][tid] - M);
        gm[tid] = M;
        gl[tid] = l;
    }
    for (int i = tid; i < GP * kD; i += kThreads) {
        const int g = i / kD, j = i % kD;
        float M = -INFINITY;
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wm[w][g]);
        float acc_i = 0.f;
        for (int w = 0; w < kWaves; ++w)
            if (wm[w][g] != -INFINITY) acc_i += wacc[w][g][j] * exp2f(wm[w][g] - M);
        rot[i] = acc_i;
    }
    __syncthreads();
    for (int hh = 1; hh < kD; hh <<= 1) {
        for (int i = tid; i < GP * (kD / 2); i += kThreads) {
            const int g = i / (kD / 2), x = i % (kD / 2);
            const int lo = (x / hh) * 2 * hh + (x % hh);
            const float x0 = rot[g * kD + lo], x1 = rot[g * kD + lo + hh];
            rot[g * kD + lo] = x0 + x1;
            rot[g * kD + lo + hh] = x0 - x1;
        }
        __syncthreads();
    }
    for (int i = tid; i < G * kD; i += kThreads) {
        const int g = i / kD, j = i % kD;
        const int64_t slot = ((int64_t)b * a.Hq + hq0 + g) * (NC + kResSlots) + c;
        a.ws_acc[slot * kD + j] = rot[i];
        if (j == 0) {
            a.ws_m[slot] = gm[g];
            a.ws_l[slot] = gl[g];
        }
    }
}

}  // namespace

// Chunks: about six workgroups per CU but at most 64 chunks per sequence
// (the merge reads up to 64 partials in one pass, one per lane), in whole
// workgroup passes of 128 tokens, at least kMinChunkHead and at most kMaxChunkB
// tokens.
int launch_bf16_partial(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, const uint16_t* k,
                        const uint16_t* v, const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                        hipStream_t stream) {
    const int64_t pairs = (int64_t)B * Hkv;
    int64_t nc = std::max<int64_t>((t_cap + kMaxChunkB - 1) / kMaxChunkB,
                                   std::min<int64_t>((6 * cu_count() + pairs - 1) / pairs, 64));
    int chunk = (int)((t_cap + nc - 1) / nc);
    chunk = std::max(((chunk + kPass - 1) / kPass) * kPass, kMinChunkHead);
    B16Args a;
    a.q = q;
    a.k = k;
    a.v = v;
    a.seq_lens = seq_lens;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = Hq / Hkv;
    a.t_cap = t_cap;
    a.chunk = chunk;
    a.nchunks = (t_cap + chunk - 1) / chunk;
    a.scale_log2 = scale * 1.4426950408889634f;
    const int64_t slots = ws_slots(B, Hq, t_cap);
    a.ws_hdr = static_cast<int32_t*>(ws);
    a.ws_acc = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsHeader);
    a.ws_m = a.ws_acc + slots * kD;
    a.ws_l = a.ws_m + slots;
    const dim3 grid(a.nchunks, Hkv, B);
    if (a.G <= 4)
        bf16_partial_kernel<4><<<grid, kThreads, 0, stream>>>(a);
    else
        bf16_partial_kernel<8><<<grid, kThreads, 0, stream>>>(a);
    return hip_check("bf16_partial launch", hipGetLastError());
}

}  // namespace dq
