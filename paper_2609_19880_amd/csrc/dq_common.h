// Device helpers shared by the kernels.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dq_internal.h"

namespace dq {

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ float half_bits_to_f32(uint16_t h) {
    return __half2float(__ushort_as_half(h));
}

// LDS visibility between lanes of one wavefront.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wavefront reductions on the DPP network (no LDS traffic).  Quad
// permutations and row mirrors reduce each row of 16 lanes; two row broadcasts
// carry the row results up to lane 63, which is read back as a uniform value.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, ROW_MASK, 0xF, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_step(float v) {
    return __uint_as_float(dpp_u32<CTRL, ROW_MASK>(__float_as_uint(v)));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_step(int v) {
    return (int)dpp_u32<CTRL, ROW_MASK>((uint32_t)v);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_step(double v) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint64_t lo = dpp_u32<CTRL, ROW_MASK>((uint32_t)u);
    const uint64_t hi = dpp_u32<CTRL, ROW_MASK>((uint32_t)(u >> 32));
    return __longlong_as_double((long long)(lo | (hi << 32)));
}

__device__ __forceinline__ float lane63(float v) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ int lane63(int v) { return __builtin_amdgcn_readlane(v, 63); }
__device__ __forceinline__ double lane63(double v) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
    return __longlong_as_double((long long)(lo | (hi << 32)));
}

template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
    v = op(v, dpp_step<0xB1, 0xF>(v));    // quad_perm [1, 0, 3, 2]
    v = op(v, dpp_step<0x4E, 0xF>(v));    // quad_perm [2, 3, 0, 1]
    v = op(v, dpp_step<0x141, 0xF>(v));   // row_half_mirror
    v = op(v, dpp_step<0x140, 0xF>(v));   // row_mirror: every lane holds its row's result
    v = op(v, dpp_step<0x142, 0xA>(v));   // row_bcast:15 into rows 1 and 3
    v = op(v, dpp_step<0x143, 0xC>(v));   // row_bcast:31 into rows 2 and 3
    return lane63(v);
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
    return wave_reduce(v, [](T a, T b) { return a > b ? a : b; });
}

template <typename T>
__device__ __forceinline__ T wave_min(T v) {
    return wave_reduce(v, [](T a, T b) { return a < b ? a : b; });
}

// Sums: the lanes a row mask leaves out take 0 instead of their own value,
// which lets each step be one add with a DPP source.  The lanes read at the
// end (lane 63's row) see the same additions in the same order either way.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp0_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xF, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp0(int v) { return (int)dpp0_u32<CTRL, ROW_MASK>((uint32_t)v); }
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp0(float v) { return __uint_as_float(dpp0_u32<CTRL, ROW_MASK>(__float_as_uint(v))); }

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
    v += dpp0<0xB1, 0xF>(v);
    v += dpp0<0x4E, 0xF>(v);
    v += dpp0<0x141, 0xF>(v);
    v += dpp0<0x140, 0xF>(v);
    v += dpp0<0x142, 0xA>(v);
    v += dpp0<0x143, 0xC>(v);
    return lane63(v);
}

// Sum over each half-wavefront: lanes 16-31 end with the sum of lanes 0-31,
// lanes 48-63 with that of lanes 32-63.
__device__ __forceinline__ float half_sum_f32(float v) {
    v += dpp0<0xB1, 0xF>(v);    // quad_perm [1, 0, 3, 2]
    v += dpp0<0x4E, 0xF>(v);    // quad_perm [2, 3, 0, 1]
    v += dpp0<0x141, 0xF>(v);   // row_half_mirror
    v += dpp0<0x140, 0xF>(v);   // row_mirror: every lane holds its row's sum
    v += dpp0<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
    return v;
}

// v of lane l ^ HH (HH a power of two below 64) with no LDS traffic: DPP
// within rows of 16 lanes, the gfx950 lane-swap instructions across them.
template <int HH>
__device__ __forceinline__ float xor_lane(float v, int lane) {
    const int x = __float_as_int(v);
    if constexpr (HH == 1) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));     // quad_perm [1,0,3,2]
    } else if constexpr (HH == 2) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));     // quad_perm [2,3,0,1]
    } else if constexpr (HH == 4) {
        // lanes with bit 2 clear (banks 0 and 2 of a row) read l + 4 (row_ror:12),
        // the others l - 4 (row_ror:4)
        int t = __builtin_amdgcn_update_dpp(0, x, 0x12C, 0xF, 0x5, false);
        t = __builtin_amdgcn_update_dpp(t, x, 0x124, 0xF, 0xA, false);
        return __int_as_float(t);
    } else if constexpr (HH == 8) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false));    // row_ror:8
    } else if constexpr (HH == 16) {
        // odd rows of the first result hold the even rows of the source and
        // even rows of the second the odd rows
        const auto r = __builtin_amdgcn_permlane16_swap((unsigned)x, (unsigned)x, false, false);
        return __uint_as_float((lane & 16) ? r[0] : r[1]);
    } else {
        static_assert(HH == 32, "xor_lane: HH in 1, 2, 4, ..., 32");
        const auto r = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
        return __uint_as_float((lane & 32) ? r[0] : r[1]);
    }
}

template <int HH>
__device__ __forceinline__ void hadamard_stage(float& v0, float& v1, int lane) {
    const float p0 = xor_lane<HH>(v0, lane), p1 = xor_lane<HH>(v1, lane);
    v0 = (lane & HH) ? p0 - v0 : v0 + p0;
    v1 = (lane & HH) ? p1 - v1 : v1 + p1;
}

// Stages h = 1, 2, ..., 32 of the unnormalized Hadamard transform of a
// 128-vector held as channels l (v0) and l + 64 (v1) in lane l, in the order
// of the definition; stage 64 is (v0 + v1, v0 - v1), left to the caller.
__device__ __forceinline__ void hadamard_lanes(float& v0, float& v1, int lane) {
    hadamard_stage<1>(v0, v1, lane);
    hadamard_stage<2>(v0, v1, lane);
    hadamard_stage<4>(v0, v1, lane);
    hadamard_stage<8>(v0, v1, lane);
    hadamard_stage<16>(v0, v1, lane);
    hadamard_stage<32>(v0, v1, lane);
}

__device__ __forceinline__ int wave_sum_i32(int v) { return wave_sum(v); }

__device__ __forceinline__ float wave_sum_f32(float v) { return wave_sum(v); }

// Maximum of non-NaN floats (the sign of a zero result is unspecified), one
// v_max_f32 with a DPP source per step.  The DPP operand's wait states after a
// VALU write (and after a VALU write of EXEC) are issued here, since the
// compiler does not look inside the statements.
__device__ __forceinline__ float wave_max_f32(float v) {
    asm("s_nop 4\n\t"
        "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "s_nop 1"
        : "+v"(v));
    return lane63(v);
}

// wave_max_f32 of four values at once: the four DPP chains are interleaved,
// so each step's operand is written three instructions before it is read
// (no wait states to pad).
__device__ __forceinline__ void wave_max4_f32(float (&v)[4]) {
    asm("s_nop 4\n\t"
        "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %0, %0, %0 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %0, %0, %0 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "v_max_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "v_max_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "v_max_f32_dpp %1, %1, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "v_max_f32_dpp %2, %2, %2 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "v_max_f32_dpp %3, %3, %3 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "s_nop 1"
        : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = lane63(v[k]);
}

}  // namespace dq
