// BF16 decode attention over an uncompressed cache: the comparator of the
// compressed path, on the same shapes (K and V bf16 [B][Hkv][t_cap][d] in the
// original basis), writing the same split-K partials so that attn_merge_kernel
// finishes it.  It is the textbook computation the residual window does for a
// few tokens, at full context; a step reads 2 x 256 bytes per (token, KV head)
// instead of the records' 72.
//
// One workgroup per (chunk, KV head, sequence), 8 wavefronts over 64-token
// tiles.  Logits: lane = token, the 256-byte key row loaded whole and dotted
// with the G query heads held in LDS.  Values: lane = channel pair, one
// 256-byte row per load instruction (coalesced), weights broadcast from LDS.
// The chunk's value sum is rotated (H acc) before it is stored, since the
// merge undoes the rotation of the compressed path (H H = d I).
#include <math.h>

#include <algorithm>

#include "dq_common.h"

namespace dq {
namespace {

constexpr int kD = 128;
constexpr int kTile = 64;
constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kMaxChunkB = 16384;

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

template <int GP>
__global__ __launch_bounds__(kThreads) void bf16_partial_kernel(B16Args a) {
    __shared__ __align__(16) float qs[GP][kD];
    __shared__ float pw[kWaves][GP][kTile];
    __shared__ float wm[kWaves][GP], wl[kWaves][GP];
    __shared__ float wacc[kWaves][GP][kD];
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
    for (int i = tid; i < GP * kD; i += kThreads) {
        const int g = i / kD;
        qs[g][i % kD] = g < G ? bf16_to_f32(a.q[((int64_t)b * a.Hq + hq0) * kD + i]) : 0.f;
    }
    __syncthreads();

    const int64_t row0 = ((int64_t)b * a.Hkv + h) * a.t_cap;
    float m_run[GP], l_part[GP], acc0[GP], acc1[GP];
#pragma unroll
    for (int g = 0; g < GP; ++g) {
        m_run[g] = -INFINITY;
        l_part[g] = 0.f;
        acc0[g] = acc1[g] = 0.f;
    }
    const int ntiles = (min(a.chunk, T - start) + kTile - 1) / kTile;
    for (int tile = wave; tile < ntiles; tile += kWaves) {
        const int t_base = start + tile * kTile;
        const int t = t_base + lane;               // < t_cap: tiles lie inside the capacity
        const bool valid = t < T;
        // ---- logits, lane = token
        const uint4* kp = reinterpret_cast<const uint4*>(a.k + (row0 + t) * kD);
        uint4 kr[kD / 8];
#pragma unroll
        for (int c8 = 0; c8 < kD / 8; ++c8) kr[c8] = kp[c8];
        float dot[GP];
#pragma unroll
        for (int g = 0; g < GP; ++g) dot[g] = 0.f;
#pragma unroll
        for (int c8 = 0; c8 < kD / 8; ++c8) {
            const uint32_t ww[4] = {kr[c8].x, kr[c8].y, kr[c8].z, kr[c8].w};
#pragma unroll
            for (int g = 0; g < GP; ++g) {
                const float4 qa = *reinterpret_cast<const float4*>(&qs[g][c8 * 8]);
                const float4 qb = *reinterpret_cast<const float4*>(&qs[g][c8 * 8 + 4]);
                const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    dot[g] += qv[e] * __uint_as_float((e & 1) ? (ww[e >> 1] & 0xFFFF0000u) : (ww[e >> 1] << 16));
            }
        }
        // ---- online softmax per head
#pragma unroll
        for (int g = 0; g < GP; ++g) {
            const float s = (valid && g < G) ? dot[g] * a.scale_log2 : -INFINITY;
            const float mn = fmaxf(m_run[g], wave_max_f32(s));
            const float corr = (m_run[g] == -INFINITY || mn == -INFINITY) ? (m_run[g] == mn ? 1.f : 0.f)
                                                                           : __builtin_amdgcn_exp2f(m_run[g] - mn);
            const float p = s == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s - mn);
            l_part[g] = l_part[g] * corr + p;
            acc0[g] *= corr;
            acc1[g] *= corr;
            m_run[g] = mn;
            pw[wave][g][lane] = p;
        }
        wave_sync();
        // ---- weighted values, lane = channel pair; 16 rows in flight at a time
        for (int u0 = 0; u0 < kTile; u0 += 16) {
            uint32_t vw[16];
#pragma unroll
            for (int u = 0; u < 16; ++u)
                vw[u] = *reinterpret_cast<const uint32_t*>(a.v + (row0 + t_base + u0 + u) * kD + 2 * lane);
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const float v0 = __uint_as_float(vw[u] << 16), v1 = __uint_as_float(vw[u] & 0xFFFF0000u);
#pragma unroll
                for (int g = 0; g < GP; ++g) {
                    const float p = pw[wave][g][u0 + u];
                    acc0[g] += p * v0;
                    acc1[g] += p * v1;
                }
            }
        }
        wave_sync();    // pw is rewritten by the next tile
    }

    // ---- merge the wavefronts, rotate, store the chunk's partial
#pragma unroll
    for (int g = 0; g < GP; ++g) {
        const float l = wave_sum_f32(l_part[g]);
        if (lane == 0) {
            wm[wave][g] = m_run[g];
            wl[wave][g] = l;
        }
        wacc[wave][g][2 * lane] = acc0[g];
        wacc[wave][g][2 * lane + 1] = acc1[g];
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
        float acc = 0.f;
        for (int w = 0; w < kWaves; ++w)
            if (wm[w][g] != -INFINITY) acc += wacc[w][g][j] * exp2f(wm[w][g] - M);
        rot[i] = acc;
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

// Chunks: about three workgroups per CU (a workgroup holds 8 wavefronts), in
// whole passes of 512 tokens, at most kMaxChunkB tokens.
int launch_bf16_partial(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, const uint16_t* k,
                        const uint16_t* v, const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                        hipStream_t stream) {
    const int64_t pairs = (int64_t)B * Hkv;
    const int pass = kWaves * kTile;
    int64_t nc = std::max<int64_t>((t_cap + kMaxChunkB - 1) / kMaxChunkB, (3 * cu_count() + pairs - 1) / pairs);
    int chunk = (int)((t_cap + nc - 1) / nc);
    chunk = std::max(((chunk + pass - 1) / pass) * pass, kMinChunk);
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
