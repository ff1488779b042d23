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

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i mfma(uint32_t a, uint32_t b, v4i c) {
    return __builtin_amdgcn_mfma_i32_4x4x4i8((int)a, (int)b, c, 0, 0, 0);
}

__device__ __forceinline__ float combine(const v4i& d0, const v4i& d1, const v4i& d2, int r) {
    return (float)d2[r] * 65536.0f + (float)d1[r] * 256.0f + (float)d0[r];
}

}  // namespace dq
