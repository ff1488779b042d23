// Device helpers shared by the attention kernels over D-Quant records: LDS
// addressing, fp16 header words, level packing and the int8 matrix-core
// contractions with three-digit fixed-point operands.
#pragma once

#include "dq_common.h"

namespace dq {

__device__ __forceinline__ float half_lo(uint32_t w) { return half_bits_to_f32((uint16_t)(w & 0xFFFFu)); }
__device__ __forceinline__ float half_hi(uint32_t w) { return half_bits_to_f32((uint16_t)(w >> 16)); }

// LDS access through a plain byte offset (no symbol relocation in the address).
#define LDS_PTR(T, off) reinterpret_cast<__attribute__((address_space(3))) T*>((uintptr_t)(off))

// Levels of four consecutive steps (top bytes of the table words) as one word.
__device__ __forceinline__ uint32_t pack4(uint32_t e0, uint32_t e1, uint32_t e2, uint32_t e3) {
    const uint32_t lo = __builtin_amdgcn_perm(e1, e0, 0x0c0c0703u);
    const uint32_t hi = __builtin_amdgcn_perm(e3, e2, 0x07030c0cu);
    return lo | hi;
}

// 4x4 byte transpose inside each lane quad: lane 4q+i holds row i on input
// and column i on output.
__device__ __forceinline__ uint32_t quad_transpose(uint32_t w, uint32_t sel1, uint32_t sel2) {
    const uint32_t p1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)w, 0xB1, 0xF, 0xF, false);
    const uint32_t r = __builtin_amdgcn_perm(p1, w, sel1);
    const uint32_t p2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)r, 0x4E, 0xF, 0xF, false);
    return __builtin_amdgcn_perm(p2, r, sel2);
}

// Three signed 8-bit digits of v in [-2^22, 2^22]: v = d2 2^16 + d1 2^8 + d0.
__device__ __forceinline__ void digits3(int v, int& d0, int& d1, int& d2) {
    d0 = ((v + 128) & 255) - 128;
    const int v1 = (v - d0) >> 8;
    d1 = ((v1 + 128) & 255) - 128;
    d2 = (v1 - d1) >> 8;
}

// Rotates one query head held as channels l and l + 64 in lane l
// (unnormalized Hadamard, stages h = 1, 2, ..., 64 in the order of the
// definition) and stores it into qt[g][128] fp32, with qscale[g] = max |q_rot| /
// 2^22 and qsum[g] = sum of q_rot.  rotate = 0: keys arrive in the rotated
// basis, and so does the query: it is taken as it is.  v0, v1 end as the
// rotated channels; returns qscale[g].
__device__ __forceinline__ float rotate_query_head(float& v0, float& v1, int g, int lane, float* qt, float* qscale,
                                                   float* qsum, int rotate) {
    if (rotate) {
        hadamard_lanes(v0, v1, lane);
        const float r0 = v0 + v1, r1 = v0 - v1;
        v0 = r0;
        v1 = r1;
    }
    qt[g * 128 + lane] = v0;
    qt[g * 128 + lane + 64] = v1;
    const float mx = wave_max_f32(fmaxf(fabsf(v0), fabsf(v1)));
    const float sm = wave_sum_f32(v0 + v1);
    const float qs = mx * (1.0f / 4194304.0f);
    if (lane == 0) {
        qscale[g] = qs;
        qsum[g] = sm;
    }
    return qs;
}

// All query heads of a workgroup, a wavefront per head: heads 0 .. nh - 1 of
// q, and qscale = qsum = 0 for the slots nh .. slots - 1.
__device__ __forceinline__ void rotate_query_heads(const uint16_t* q, int nh, int slots, int wave, int nw,
                                                   int lane, float* qt, float* qscale, float* qsum,
                                                   int rotate = 1) {
    for (int g = wave; g < slots; g += nw) {
        if (g >= nh) {
            if (lane == 0) {
                qscale[g] = 0.f;
                qsum[g] = 0.f;
            }
            continue;
        }
        float v0 = bf16_to_f32(q[g * 128 + lane]), v1 = bf16_to_f32(q[g * 128 + lane + 64]);
        rotate_query_head(v0, v1, g, lane, qt, qscale, qsum, rotate);
    }
}

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i mfma(uint32_t a, uint32_t b, v4i c) {
    return __builtin_amdgcn_mfma_i32_4x4x4i8((int)a, (int)b, c, 0, 0, 0);
}

// v_mfma_i32_16x16x32_i8: lane l gives row l % 16 and K = 8 (l / 16) .. + 7
// of A, the same K of column l % 16 of B, and receives rows 4 (l / 16) .. + 3
// of column l % 16.
__device__ __forceinline__ v4i mfma16(uint64_t a, uint64_t b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x32_i8((long)a, (long)b, c, 0, 0, 0);
}

// ds_read_b64_tr_b8 at LDS byte address off.  Within each group of 16 lanes,
// lane 8 h + i receives byte i of the 8-byte rows that the group's lanes h,
// h + 2, ..., h + 14 address (in that order): token-major rows come back
// K-major, as the 16x16x32 products take them.
__device__ __forceinline__ uint64_t lds_tr8(uint32_t off) {
    typedef int v2i __attribute__((ext_vector_type(2)));
    const v2i r = __builtin_amdgcn_ds_read_tr8_b64_v2i32(LDS_PTR(v2i, off));
    return (uint64_t)(uint32_t)r.x | ((uint64_t)(uint32_t)r.y << 32);
}

// v[slot] for slot in 0..3 (v held in registers, slot per lane).
__device__ __forceinline__ float pick4(const float* v, int slot) {
    return slot == 0 ? v[0] : slot == 1 ? v[1] : slot == 2 ? v[2] : v[3];
}

__device__ __forceinline__ float combine(const v4i& d0, const v4i& d1, const v4i& d2, int r) {
    return (float)d2[r] * 65536.0f + (float)d1[r] * 256.0f + (float)d0[r];
}

}  // namespace dq
