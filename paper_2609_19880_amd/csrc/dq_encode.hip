// Append path: bf16 K/V tokens -> fixed-size D-Quant records (Fig. 1, Alg. 1).
//
// Two kernels:
//  * key_mean: one wavefront per (batch, head, 128-token window).  Rotates
//    each token (Hadamard, Sec. 4.2), sums the window left to right in fp64,
//    and stores the channel mean as INT8 with one fp16 scale (Sec. 4.2,
//    App. B).
//  * encode: one workgroup per (batch, head, 64 consecutive tokens; 32 for
//    per-token streams).  Each wavefront takes a stream at a time with its n
//    values spread over the lanes and keeps them in registers through Alg. 1
//    (FitMinMax -> Drift -> Refit -> fp16 -> Drift); no n x M distortion
//    matrix goes to memory (the distortions of up to 8 or 16 levels stay in
//    registers for the assignments of a drift, more levels are recomputed on
//    the fly) and the code length is reduced across the wavefront, as
//    Sec. 4.5 describes for the encoder.  The symbols of the workgroup's
//    streams then go through LDS to lane-per-stream backward rANS (divisions
//    by f as exact multiply-high reciprocals), and the records are written as
//    one contiguous span.
//
// Every floating-point step is fp64 in a fixed order without contraction
// (this file is built with -ffp-contract=off), so the records are
// bit-identical to the reference definition of the format.
#include <float.h>
#include <limits.h>

#include "dq_common.h"

namespace dq {
namespace {

constexpr int kEncStreams = 64;   // streams per workgroup
// Per-token streams (n = 1024) stage 32: their symbols and records then take
// about 48 KB of LDS, so that three workgroups share a CU (64 streams would
// leave one wavefront per SIMD).
constexpr int kEncStreamsTok = 32;
__host__ __device__ constexpr int enc_streams(bool tok) { return tok ? kEncStreamsTok : kEncStreams; }
constexpr int kEncWaves = 4;
constexpr int kEncThreads = kEncWaves * kWave;
constexpr int kD = 128;           // head_dim of the heads in a per-token stream

// Unnormalized FWHT of each group of 64 * SPAN values (a whole stream, or one
// attention head of a per-token stream); lane l holds elements l + 64 k, group
// k / SPAN.  Stages run h = 1, 2, ..., 32 SPAN as in the definition.
template <int VPL, int SPAN = VPL>
__device__ __forceinline__ void fwht_wave(double (&v)[VPL], int lane) {
#pragma unroll
    for (int h = 1; h < kWave; h <<= 1) {
#pragma unroll
        for (int k = 0; k < VPL; ++k) {
            double pv = __shfl_xor(v[k], h);
            v[k] = (lane & h) ? (pv - v[k]) : (v[k] + pv);
        }
    }
#pragma unroll
    for (int s = 1; s < SPAN; s <<= 1) {
#pragma unroll
        for (int k = 0; k < VPL; ++k) {
            if (!(k & s)) {
                double a = v[k], b = v[k + s];
                v[k] = a + b;
                v[k + s] = a - b;
            }
        }
    }
}

// Fold-in-halves sum of the n = 64 VPL values (v[i] += v[i + len/2] until
// one is left); every lane ends with the total.
template <int VPL>
__device__ __forceinline__ double fold_sum(const double (&v)[VPL]) {
    double w[VPL];
#pragma unroll
    for (int k = 0; k < VPL; ++k) w[k] = v[k];
#pragma unroll
    for (int len = VPL; len > 1; len >>= 1) {
#pragma unroll
        for (int k = 0; k < len / 2; ++k) w[k] = w[k] + w[k + len / 2];
    }
    double s = w[0];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s = s + __shfl_xor(s, off);
    return s;
}

// rotate = 0: the input is already in the rotated basis (prerotated tables).
template <int VPL>
__device__ __forceinline__ void load_rotated(const uint16_t* src, double (&v)[VPL], int lane, int rotate) {
#pragma unroll
    for (int k = 0; k < VPL; ++k) v[k] = (double)bf16_to_f32(src[lane + kWave * k]);
    if (rotate) fwht_wave<VPL>(v, lane);
}

// Per-token stream (head_dim 128): head g's channels c = lane + 64 i are
// elements k = 2 g + i, each head rotated on its own.
template <int VPL>
__device__ __forceinline__ void load_token_rotated(const uint16_t* src, int64_t sh, double (&v)[VPL], int lane,
                                                   int rotate) {
#pragma unroll
    for (int k = 0; k < VPL; ++k) v[k] = (double)bf16_to_f32(src[(int64_t)(k / 2) * sh + lane + kWave * (k % 2)]);
    if (rotate) fwht_wave<VPL, 2>(v, lane);
}

struct DriftCtx {
    const double* rate;    // LDS [M]: R_m / 2^16
    const int32_t* cost;   // LDS [M]
    const float* lam;      // LDS [512]
    int M;
    int cheapest;
    int rmin;
};

// max / min of two non-NaN doubles as one v_max_f64 / v_min_f64 (fmax and
// fmin would first quiet possible signalling NaNs, one more instruction per
// operand).  Distortions and penalties are >= +0, so which of two equal zeros
// comes out never matters.
__device__ __forceinline__ double max_nn(double a, double b) {
    double r;
    asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ double min_nn(double a, double b) {
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// DPP copy of a double; lanes that a row mask leaves out are undefined, which
// a reduction read back from lane 63 never sees.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_copy(double v) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint64_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, ROW_MASK, 0xF, false);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, ROW_MASK, 0xF, false);
    return __longlong_as_double((long long)(lo | (hi << 32)));
}

// Wavefront max / min of non-NaN doubles with no -0 (the distortions).
template <bool MAX>
__device__ __forceinline__ double wave_ext_nn(double v) {
    auto op = [](double a, double b) { return MAX ? max_nn(a, b) : min_nn(a, b); };
    v = op(v, dpp_copy<0xB1, 0xF>(v));
    v = op(v, dpp_copy<0x4E, 0xF>(v));
    v = op(v, dpp_copy<0x141, 0xF>(v));
    v = op(v, dpp_copy<0x140, 0xF>(v));
    v = op(v, dpp_copy<0x142, 0xA>(v));
    v = op(v, dpp_copy<0x143, 0xC>(v));
    return lane63(v);
}

// Assignment at one lambda: each value takes argmin_m D_im + lambda r_m (ties to
// the smallest m); returns the wavefront's total Q16 cost.  MB > 0: the
// distortions D[k][m] of the M <= MB levels were computed once per drift;
// MB = 0: they are recomputed here (t = s m, u = o + t, e = x - u, D = e e).
// rt: the rates R_m / 2^16 of the MB levels in registers (MB > 0).
template <int VPL, int MB>
__device__ __forceinline__ int assign_cost(const double (&x)[VPL], const double (&D)[VPL][MB > 0 ? MB : 1],
                                           const double (&rt)[MB > 0 ? MB : 1], double s, double o,
                                           double lam, const DriftCtx& c, int (&m)[VPL]) {
    double best[VPL];
    if (MB > 0) {
        const double pen0 = lam * rt[0];
#pragma unroll
        for (int k = 0; k < VPL; ++k) {
            best[k] = D[k][0] + pen0;
            m[k] = 0;
        }
#pragma unroll
        for (int mm = 1; mm < (MB > 0 ? MB : 1); ++mm) {
            if (mm < c.M) {
                const double pen = lam * rt[mm];
#pragma unroll
                for (int k = 0; k < VPL; ++k) {
                    const double J = D[k][mm] + pen;
                    m[k] = J < best[k] ? mm : m[k];
                    best[k] = min_nn(best[k], J);
                }
            }
        }
    } else {
        {
            const double t = s * 0.0;
            const double u = o + t;
            const double pen = lam * c.rate[0];
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const double e = x[k] - u;
                best[k] = e * e + pen;
                m[k] = 0;
            }
        }
        for (int mm = 1; mm < c.M; ++mm) {
            const double t = s * (double)mm;
            const double u = o + t;
            const double pen = lam * c.rate[mm];
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const double e = x[k] - u;
                const double J = e * e + pen;
                m[k] = J < best[k] ? mm : m[k];
                best[k] = min_nn(best[k], J);
            }
        }
    }
    int cst = 0;
#pragma unroll
    for (int k = 0; k < VPL; ++k) cst += c.cost[m[k]];
    return wave_sum_i32(cst);
}

// Drift(x, s, o, r, B) of Alg. 1: bisection on log2(lambda) over a
// 40-octave bracket below hi = ceil(log2(8 (max D - min D))), lambda on the
// 2^(U/512) grid, 12 steps, assignment at the final hi; nearest cheapest
// symbol if even that overflows; cheapest symbol if all distortions are equal.
template <int VPL, int MB>
__device__ void drift(const double (&x)[VPL], double s, double o, int64_t budget,
                      const DriftCtx& c, int (&m)[VPL]) {
    double D[VPL][MB > 0 ? MB : 1], rt[MB > 0 ? MB : 1];
    double dmax = -DBL_MAX, dmin = DBL_MAX;
    if (MB > 0) {
#pragma unroll
        for (int mm = 0; mm < (MB > 0 ? MB : 1); ++mm) {
            rt[mm] = mm < c.M ? c.rate[mm] : 0.0;
            const double t = s * (double)mm;
            const double u = o + t;
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const double e = x[k] - u;
                D[k][mm] = e * e;
                if (mm < c.M) {
                    dmax = max_nn(dmax, D[k][mm]);
                    dmin = min_nn(dmin, D[k][mm]);
                }
            }
        }
    } else {
        for (int mm = 0; mm < c.M; ++mm) {
            const double t = s * (double)mm;
            const double u = o + t;
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const double e = x[k] - u;
                const double Dv = e * e;
                dmax = max_nn(dmax, Dv);
                dmin = min_nn(dmin, Dv);
            }
        }
    }
    dmax = wave_ext_nn<true>(dmax);
    dmin = wave_ext_nn<false>(dmin);
    if (dmax == dmin) {
#pragma unroll
        for (int k = 0; k < VPL; ++k) m[k] = c.cheapest;
        return;
    }
    int ex = 0;
    const double mant = frexp(8.0 * (dmax - dmin), &ex);
    const int hi = (mant == 0.5) ? ex - 1 : ex;
    int u_hi = hi * kLambdaSteps;
    int u_lo = u_hi - kBracketUnits;
    // the code length is an int: comparing it with the budget clamped to
    // INT_MAX decides the same and stays a scalar compare
    const int budget32 = (int)(budget < INT_MAX ? budget : INT_MAX);
    // m holds the assignment at u_hi once a step has moved u_hi: the final
    // assignment at u_hi is then that step's, and within the budget.  With 16
    // values per lane the copy's registers cost more occupancy than the
    // final assignment it saves, which is then recomputed.
    constexpr bool kKeepHi = VPL <= 4;
    bool at_hi = false;
    for (int it = 0; it < kBisectSteps; ++it) {
        const int u_mid = (u_lo + u_hi) >> 1;
        const double lam = ldexp((double)c.lam[u_mid & (kLambdaSteps - 1)], u_mid >> 9);
        int tmp[VPL];
        const int cst = assign_cost<VPL, MB>(x, D, rt, s, o, lam, c, tmp);
        if (cst <= budget32) {
            u_hi = u_mid;
            if (kKeepHi) {
                at_hi = true;
#pragma unroll
                for (int k = 0; k < VPL; ++k) m[k] = tmp[k];
            }
        } else {
            u_lo = u_mid;
        }
    }
    if (at_hi) return;
    const double lam = ldexp((double)c.lam[u_hi & (kLambdaSteps - 1)], u_hi >> 9);
    const int cst = assign_cost<VPL, MB>(x, D, rt, s, o, lam, c, m);
    if (cst > budget32) {
        double best[VPL];
#pragma unroll
        for (int k = 0; k < VPL; ++k) best[k] = DBL_MAX;
        for (int mm = 0; mm < c.M; ++mm) {
            if (c.cost[mm] != c.rmin) continue;
            const double t = s * (double)mm;
            const double u = o + t;
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const double e = x[k] - u;
                const double Dv = e * e;
                if (Dv < best[k]) {
                    best[k] = Dv;
                    m[k] = mm;
                }
            }
        }
    }
}

__device__ __forceinline__ uint16_t f64_to_half_bits(double v) {
    return __half_as_ushort(__float2half_rn((float)v));
}

template <int VPL>
__global__ __launch_bounds__(kWave) void key_mean_kernel(const uint16_t* __restrict__ kv,
                                                         int64_t sb, int64_t st, int64_t sh, int H,
                                                         int t0, int t_cap, Pages pg,
                                                         int8_t* __restrict__ mean_q,
                                                         uint16_t* __restrict__ mean_scale,
                                                         uint32_t* status, int rotate) {
    constexpr int n = kWave * VPL;
    const int w = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x;
    double acc[VPL];
#pragma unroll
    for (int k = 0; k < VPL; ++k) acc[k] = 0.0;
    const uint16_t* base = kv + (int64_t)b * sb + (int64_t)h * sh;
    const int tw = w * DQ_MEAN_WINDOW;
    for (int t = 0; t < DQ_MEAN_WINDOW; ++t) {
        double v[VPL];
        load_rotated<VPL>(base + (int64_t)(tw + t) * st, v, lane, rotate);
#pragma unroll
        for (int k = 0; k < VPL; ++k) acc[k] = acc[k] + v[k];
    }
    double mu[VPL];
    double amax = 0.0;
    bool finite = true;
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
        mu[k] = acc[k] / (double)DQ_MEAN_WINDOW;
        amax = fmax(amax, fabs(mu[k]));
        finite = finite && isfinite(mu[k]);
    }
    amax = wave_max(amax);
    const uint16_t sbits = f64_to_half_bits(amax / 127.0);
    const double sc = (double)__half2float(__ushort_as_half(sbits));
    bool bad_page = false;
    const int64_t widx = window_index(pg, H, t_cap, b, h, t0 / DQ_MEAN_WINDOW + w, bad_page);
    if (bad_page) {             // nothing is written through a block-table entry outside the pool
        if (lane == 0 && status) atomicOr(status, DQ_STATUS_PAGE);
        return;
    }
    int8_t* dst = mean_q + widx * n;
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
        double qv = 0.0;
        if (sc > 0.0) qv = fmin(127.0, fmax(-127.0, rint(mu[k] / sc)));
        dst[lane + kWave * k] = (int8_t)qv;
    }
    if (lane == 0) mean_scale[widx] = sbits;
    const bool bad = __any(!finite) || !isfinite(sc);
    if (bad && lane == 0 && status) atomicOr(status, DQ_STATUS_RANGE);
}

struct EncArgs {
    TabArgs ta;
    const uint16_t* kv;
    int64_t sb, st, sh;
    int H, t0, n_new, t_cap;
    Pages pg;                    // records and key means: contiguous or paged
    int rec_stride;              // per-token records: bytes per record slot (multiple of 16)
    uint8_t* records;
    const int8_t* mean_q;        // NULL for values
    const uint16_t* mean_scale;
    uint32_t* status;
    int rotate;                  // 0: the input is already in the rotated basis
};

// x = rotated stream of cache token t minus the dequantized window mean (keys).
// TOK: the stream spans every KV head (head g in elements 2 g, 2 g + 1).
template <int VPL, bool TOK>
__device__ __forceinline__ void stream_values(const EncArgs& a, int b, int h, int t,
                                              double (&x)[VPL], int lane) {
    const int64_t ti = t - a.t0;   // position in the input
    if (TOK) {
        load_token_rotated<VPL>(a.kv + (int64_t)b * a.sb + ti * a.st, a.sh, x, lane, a.rotate);
        if (a.mean_q) {
            bool bad = false;      // (a bad entry reads page 0; the record write then skips it)
#pragma unroll
            for (int g = 0; g < VPL / 2; ++g) {
                const int64_t wi = window_index(a.pg, a.H, a.t_cap, b, g, t / DQ_MEAN_WINDOW, bad);
                const double sc = (double)__half2float(__ushort_as_half(a.mean_scale[wi]));
                const int8_t* mq = a.mean_q + wi * kD;
                x[2 * g] = x[2 * g] - sc * (double)mq[lane];
                x[2 * g + 1] = x[2 * g + 1] - sc * (double)mq[lane + kWave];
            }
        }
        return;
    }
    load_rotated<VPL>(a.kv + (int64_t)b * a.sb + ti * a.st + (int64_t)h * a.sh, x, lane, a.rotate);
    if (a.mean_q) {
        constexpr int n = kWave * VPL;
        bool bad = false;          // (a bad entry reads page 0; the record write then skips it)
        const int64_t wi = window_index(a.pg, a.H, a.t_cap, b, h, t / DQ_MEAN_WINDOW, bad);
        const double sc = (double)__half2float(__ushort_as_half(a.mean_scale[wi]));
        const int8_t* mq = a.mean_q + wi * n;
#pragma unroll
        for (int k = 0; k < VPL; ++k) x[k] = x[k] - sc * (double)mq[lane + kWave * k];
    }
}

// Nearest level on the grid (o, s): argmin_m (x - (o + s m))^2, the same
// arithmetic as the distortions of a drift, ties to the smallest m.
template <int VPL>
__device__ __forceinline__ void nearest(const double (&x)[VPL], double s, double o, int M, int (&m)[VPL]) {
    double best[VPL];
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
        best[k] = DBL_MAX;
        m[k] = 0;
    }
    for (int mm = 0; mm < M; ++mm) {
        const double t = s * (double)mm;
        const double u = o + t;
#pragma unroll
        for (int k = 0; k < VPL; ++k) {
            const double e = x[k] - u;
            const double D = e * e;
            if (D < best[k] || mm == 0) {
                best[k] = D;
                m[k] = mm;
            }
        }
    }
}

// FIXED: the fixed-width comparator of App. B -- the same preprocessing and
// refit with nearest-level rounding in place of both drifts, and b-bit
// symbols (M = 2^b, b = 8 (C - 4) / n rounded down) packed after the 4-byte
// header, least significant bit first, instead of the rANS payload.
// Per-token streams and 16 levels in registers: three workgroups per CU (at
// most 168 VGPRs; the per-token LDS staging, about 48 KB, fits three).
template <int VPL, int MB, bool TOK, bool FIXED = false>
__global__ __launch_bounds__(kEncThreads, (TOK || MB == 16) ? 3 : 1) void encode_kernel(EncArgs a) {
    constexpr int n = kWave * VPL;
    constexpr int NS = enc_streams(TOK);
    extern __shared__ __align__(16) uint8_t smem[];
    // layout: rate[64] f64 | cost[64] | lam[512] | budget[64] i64 | s16[64] | o16[64]
    //         | flag[64] | (f, c, rcp, rsh)[64] | sym[64][n] | rec[64][C]
    double* s_rate = reinterpret_cast<double*>(smem);
    int32_t* s_cost = reinterpret_cast<int32_t*>(s_rate + DQ_MAX_LEVELS);
    float* s_lam = reinterpret_cast<float*>(s_cost + DQ_MAX_LEVELS);
    int64_t* s_budget = reinterpret_cast<int64_t*>(s_lam + kLambdaSteps);
    uint16_t* s_s16 = reinterpret_cast<uint16_t*>(s_budget + NS);
    uint16_t* s_o16 = s_s16 + NS;
    int32_t* s_flag = reinterpret_cast<int32_t*>(s_o16 + NS);
    uint4* s_ent = reinterpret_cast<uint4*>(s_flag + NS);     // coder entry per symbol
    uint8_t* s_sym = reinterpret_cast<uint8_t*>(s_ent + DQ_MAX_LEVELS);
    uint8_t* s_rec = s_sym + NS * n;

    const TabArgs& ta = a.ta;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int b = blockIdx.z, h = blockIdx.y;
    const int first = a.t0 + blockIdx.x * NS;
    const int active = min(NS, a.t0 + a.n_new - first);
    const int C = ta.C;

    for (int i = tid; i < (FIXED ? 0 : ta.M); i += kEncThreads) {
        s_cost[i] = ta.t.cost[i];
        s_rate[i] = (double)ta.t.cost[i] * (1.0 / 65536.0);
        // floor(x / f) = mulhi(x, rcp) >> (sh - 1) for x < 2^31, where
        // sh = ceil(log2 f) and rcp = ceil(2^(31 + sh) / f) (f = 1: x itself)
        const uint32_t f = (uint32_t)ta.t.freq[i];
        const uint32_t sh = f > 1 ? 32u - (uint32_t)__builtin_clz(f - 1u) : 0u;
        s_ent[i] = uint4{f, (uint32_t)ta.t.cum[i], f > 1 ? (uint32_t)(((1ull << (31 + sh)) + f - 1) / f) : 0u,
                         f > 1 ? sh - 1u : 0u};
    }
    for (int i = tid; i < (FIXED ? 0 : kLambdaSteps); i += kEncThreads) s_lam[i] = ta.t.lam[i];
    for (int i = tid; i < NS; i += kEncThreads) {
        s_budget[i] = ta.budget;
        s_flag[i] = 0;
    }
    __syncthreads();
    DriftCtx dc{s_rate, s_cost, s_lam, ta.M, ta.cheapest, ta.rmin};

    bool range_bad = false;
    for (int pass = 0;; ++pass) {
        // Drift, wavefront per stream.
        for (int i = wave; i < active; i += kEncWaves) {
            if (pass > 0 && !s_flag[i]) continue;
            double x[VPL];
            stream_values<VPL, TOK>(a, b, h, first + i, x, lane);
            uint16_t sb16, ob16;
            if (pass == 0) {
                double mn = x[0], mx = x[0];
                bool fin = true;
#pragma unroll
                for (int k = 0; k < VPL; ++k) {
                    mn = fmin(mn, x[k]);
                    mx = fmax(mx, x[k]);
                    fin = fin && isfinite(x[k]);
                }
                mn = wave_min(mn);
                mx = wave_max(mx);
                const double s0 = (mx - mn) / (double)(ta.M - 1);
                const double o0 = mn;
                int m1[VPL];
                if (FIXED)
                    nearest<VPL>(x, s0, o0, ta.M, m1);
                else
                    drift<VPL, MB>(x, s0, o0, ta.budget, dc, m1);
                // least-squares refit
                int sm = 0, smm = 0;
                double mx_[VPL];
#pragma unroll
                for (int k = 0; k < VPL; ++k) {
                    sm += m1[k];
                    smm += m1[k] * m1[k];
                    mx_[k] = (double)m1[k] * x[k];
                }
                sm = wave_sum_i32(sm);
                smm = wave_sum_i32(smm);
                const double Sx = fold_sum<VPL>(x);
                const double Smx = fold_sum<VPL>(mx_);
                const int64_t den_i = (int64_t)n * smm - (int64_t)sm * sm;
                double s1 = s0, o1 = o0;
                if (den_i != 0) {
                    const double den = (double)den_i;
                    const double smf = (double)sm;
                    const double s = ((double)n * Smx - smf * Sx) / den;
                    const double o = (Sx - s * smf) / (double)n;
                    if (isfinite(s) && s > 0.0) {
                        s1 = s;
                        o1 = o;
                    }
                }
                sb16 = f64_to_half_bits(s1);
                ob16 = f64_to_half_bits(o1);
                const float sf = __half2float(__ushort_as_half(sb16));
                const float of = __half2float(__ushort_as_half(ob16));
                if (__any(!fin) || !isfinite(sf) || !isfinite(of)) range_bad = true;
                if (lane == 0) {
                    s_s16[i] = sb16;
                    s_o16[i] = ob16;
                }
            } else {
                sb16 = s_s16[i];
                ob16 = s_o16[i];
            }
            const double s16 = (double)__half2float(__ushort_as_half(sb16));
            const double o16 = (double)__half2float(__ushort_as_half(ob16));
            int m2[VPL];
            if (FIXED)
                nearest<VPL>(x, s16, o16, ta.M, m2);
            else
                drift<VPL, MB>(x, s16, o16, s_budget[i], dc, m2);
#pragma unroll
            for (int k = 0; k < VPL; ++k) s_sym[i * n + lane + kWave * k] = (uint8_t)m2[k];
        }
        __syncthreads();

        if (FIXED) {
            // b-bit symbols after the header, lane per stream
            if (tid < active) {
                const int i = tid;
                uint8_t* rec = s_rec + i * C;
                const int bb = 31 - __builtin_clz(ta.M);
                for (int k = 0; k < C - 4; ++k) {
                    uint32_t v = 0;
                    for (int t = 0; t < 8; ++t) {
                        const int g = 8 * k + t, j = g / bb;
                        if (j < n) v |= (uint32_t)((s_sym[i * n + j] >> (g - j * bb)) & 1) << t;
                    }
                    rec[4 + k] = (uint8_t)v;
                }
                const uint16_t sb = s_s16[i], ob = s_o16[i];
                rec[0] = (uint8_t)(sb & 0xFF);
                rec[1] = (uint8_t)(sb >> 8);
                rec[2] = (uint8_t)(ob & 0xFF);
                rec[3] = (uint8_t)(ob >> 8);
            }
            __syncthreads();
            break;
        }
        // Backward rANS, lane per stream (Eq. rans, encoded in reverse).
        if (tid < active && (pass == 0 || s_flag[tid])) {
            const int i = tid;
            uint8_t* rec = s_rec + i * C;
            const int cap = C - kPayloadOffset;
            const uint32_t xmax_unit = (kRansL >> ta.p) << 8;
            uint32_t xs = kRansL;
            int emitted = 0;
            const uint32_t P = 1u << ta.p;
            for (int j = n - 1; j >= 0; --j) {
                const int m = s_sym[i * n + j];
                const uint4 ent = s_ent[m];
                const uint32_t f = ent.x, c = ent.y, rcp = ent.z, rsh = ent.w;
                const uint32_t xmax = xmax_unit * f;
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    if (xs >= xmax) {
                        if (emitted < cap) rec[C - 1 - emitted] = (uint8_t)(xs & 0xFF);
                        ++emitted;
                        xs >>= 8;
                    }
                }
                // Enc(x, m) = floor(x / f) 2^p + (x mod f) + c = x + q (2^p - f) + c;
                // after renormalization x < 256 L = 2^29
                const uint32_t q = f > 1 ? __umulhi(xs, rcp) >> rsh : xs;
                xs = xs + q * (P - f) + c;
            }
            if (emitted > cap) {
                // Defensive: with L = 2^21 the coded length is at most
                // sum r + n (2^-17 + log2(1 + 2^p / L)) bits, under 8 bits
                // past the budget for n <= 1024, so a drifted stream always
                // fits.  Should one not, retry 8 bits lower; when the budget
                // runs out the record is all zeros (decoding flags it corrupt).
                s_flag[i] = 1;
                s_budget[i] -= (int64_t)8 * 65536;
                if (s_budget[i] < (int64_t)n * ta.rmin) {
                    s_flag[i] = 0;
                    for (int k = 0; k < C; ++k) rec[k] = 0;
                    if (a.status) atomicOr(a.status, DQ_STATUS_OVERFLOW);
                }
            } else {
                s_flag[i] = 0;
                // move the payload from the end of the record to offset 8
                const int src = C - emitted;
                for (int k = 0; k < emitted; ++k) rec[kPayloadOffset + k] = rec[src + k];
                for (int k = kPayloadOffset + emitted; k < C; ++k) rec[k] = 0;
                const uint16_t sb = s_s16[i], ob = s_o16[i];
                rec[0] = (uint8_t)(sb & 0xFF);
                rec[1] = (uint8_t)(sb >> 8);
                rec[2] = (uint8_t)(ob & 0xFF);
                rec[3] = (uint8_t)(ob >> 8);
                rec[4] = (uint8_t)(xs & 0xFF);
                rec[5] = (uint8_t)((xs >> 8) & 0xFF);
                rec[6] = (uint8_t)((xs >> 16) & 0xFF);
                rec[7] = (uint8_t)(xs >> 24);
            }
        }
        const int again = __syncthreads_or(tid < active ? s_flag[tid] : 0);
        if (!again) break;
    }
    if (range_bad && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_RANGE);

    // Write the records of the active streams: one contiguous span, one record
    // at a time through the block table, or per-token records at their stride
    // (zero-padded).
    if (TOK) {
        // 64-token tiles, 8-byte chunk major: byte k of the token in row r at
        // ((r / 64) S / 8 + k / 8) 512 + (r % 64) 8 + k % 8, the row of token
        // t through the block table when there is one
        bool bad_page = false;
        for (int i = wave; i < active; i += kEncWaves) {
            const int t = first + i;
            bool bad = false;
            const int64_t row = token_row(a.pg, a.t_cap, b, t, bad);
            if (bad) {
                bad_page = true;
                continue;
            }
            uint8_t* tile = a.records + (row & ~(int64_t)63) * a.rec_stride + (row & 63) * 8;
            for (int k = lane; k < a.rec_stride; k += kWave)
                tile[(k >> 3) * 512 + (k & 7)] = k < C ? s_rec[i * C + k] : (uint8_t)0;
        }
        if (bad_page && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_PAGE);
    } else if (!a.pg.bt) {
        uint8_t* dst = a.records + ((int64_t)(b * a.H + h) * a.t_cap + first) * C;
        const int total = active * C;
        if ((((uintptr_t)dst) & 3) == 0 && (total & 3) == 0) {
            uint32_t* d32 = reinterpret_cast<uint32_t*>(dst);
            const uint32_t* s32 = reinterpret_cast<const uint32_t*>(s_rec);
            for (int k = tid; k < total / 4; k += kEncThreads) d32[k] = s32[k];
        } else {
            for (int k = tid; k < total; k += kEncThreads) dst[k] = s_rec[k];
        }
    } else {
        bool bad_page = false;
        for (int i = wave; i < active; i += kEncWaves) {
            bool bad = false;
            const int64_t row = record_row(a.pg, a.H, a.t_cap, b, h, first + i, bad);
            if (bad) {
                bad_page = true;
                continue;
            }
            uint8_t* dst = a.records + row * C;
            for (int k = lane; k < C; k += kWave) dst[k] = s_rec[i * C + k];
        }
        if (bad_page && lane == 0 && a.status) atomicOr(a.status, DQ_STATUS_PAGE);
    }
}

}  // namespace

int launch_encode(const dq_tables* tab, const Pages& pg, const uint16_t* kv, int64_t sb, int64_t st, int64_t sh,
                  int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                  uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status,
                  hipStream_t stream, int token_stride) {
    const bool tok = token_stride > 0;
    const int n = tab->cfg.head_dim;
    const int vpl = n / kWave;
    const int rotate = tab->cfg.prerotated ? 0 : 1;
    if (mean_q) {
        dim3 grid(n_new / DQ_MEAN_WINDOW, H, B);
        switch (tok ? kD / kWave : vpl) {
            case 1: key_mean_kernel<1><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, rotate); break;
            case 2: key_mean_kernel<2><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, rotate); break;
            case 4: key_mean_kernel<4><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, rotate); break;
            default: return DQ_ERR_INVALID_ARG;
        }
        if (int rc = hip_check("key_mean launch", hipGetLastError())) return rc;
    }
    EncArgs a;
    a.ta = tab_args(tab);
    a.kv = kv;
    a.sb = sb;
    a.st = st;
    a.sh = sh;
    a.H = H;
    a.t0 = t0;
    a.n_new = n_new;
    a.t_cap = t_cap;
    a.pg = pg;
    a.rec_stride = token_stride;
    a.records = records;
    a.mean_q = mean_q;
    a.mean_scale = mean_scale;
    a.status = status;
    a.rotate = rotate;
    const int ns = enc_streams(tok);
    const size_t smem = sizeof(double) * DQ_MAX_LEVELS + sizeof(int32_t) * DQ_MAX_LEVELS +
                        sizeof(float) * kLambdaSteps + sizeof(int64_t) * ns +
                        2 * sizeof(uint16_t) * ns + sizeof(int32_t) * ns +
                        sizeof(uint4) * DQ_MAX_LEVELS +
                        (size_t)ns * n + (size_t)ns * a.ta.C;
    dim3 grid((n_new + ns - 1) / ns, tok ? 1 : H, B);
    // distortions held in registers for up to 8 levels (16 with two values per
    // lane); longer streams recompute them
    const int M = tab->cfg.levels;
    const int mb = vpl > 4 ? 0 : M <= 8 ? 8 : (M <= 16 && vpl <= 2) ? 16 : 0;
    const void* fn = nullptr;
#define DQ_ENC(V, MB, T)                                                                         \
    do {                                                                                         \
        fn = reinterpret_cast<const void*>(&encode_kernel<V, MB, T>);                            \
        if (int rc = hip_check("hipFuncSetAttribute",                                            \
                               hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                                   (int)smem)))                                  \
            return rc;                                                                           \
        encode_kernel<V, MB, T><<<grid, kEncThreads, smem, stream>>>(a);                         \
    } while (0)
    switch ((tok ? 10000 : 0) + vpl * 100 + mb) {
        case 108: DQ_ENC(1, 8, false); break;
        case 116: DQ_ENC(1, 16, false); break;
        case 100: DQ_ENC(1, 0, false); break;
        case 208: DQ_ENC(2, 8, false); break;
        case 216: DQ_ENC(2, 16, false); break;
        case 200: DQ_ENC(2, 0, false); break;
        case 408: DQ_ENC(4, 8, false); break;
        case 400: DQ_ENC(4, 0, false); break;
        case 10208: DQ_ENC(2, 8, true); break;
        case 10216: DQ_ENC(2, 16, true); break;
        case 10200: DQ_ENC(2, 0, true); break;
        case 10408: DQ_ENC(4, 8, true); break;
        case 10400: DQ_ENC(4, 0, true); break;
        case 10800: DQ_ENC(8, 0, true); break;
        case 11600: DQ_ENC(16, 0, true); break;
        default: return DQ_ERR_INVALID_ARG;
    }
#undef DQ_ENC
    return hip_check("kernel launch", hipGetLastError());
}

int launch_encode_fixed(int32_t n, int32_t record_bytes, const Pages& pg, const uint16_t* kv, int64_t sb,
                        int64_t st, int64_t sh, int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                        uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status,
                        hipStream_t stream) {
    const int vpl = n / kWave;
    const int bits = 8 * (record_bytes - 4) / n;
    if (vpl < 1 || vpl > 4 || bits < 1 || bits > 8) return DQ_ERR_INVALID_ARG;
    if (mean_q) {
        dim3 grid(n_new / DQ_MEAN_WINDOW, H, B);
        switch (vpl) {
            case 1: key_mean_kernel<1><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, 1); break;
            case 2: key_mean_kernel<2><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, 1); break;
            default: key_mean_kernel<4><<<grid, kWave, 0, stream>>>(kv, sb, st, sh, H, t0, t_cap, pg, mean_q, mean_scale, status, 1); break;
        }
        if (int rc = hip_check("key_mean launch", hipGetLastError())) return rc;
    }
    EncArgs a{};
    a.ta.n = n;
    a.ta.M = 1 << bits;
    a.ta.C = record_bytes;
    a.kv = kv;
    a.sb = sb;
    a.st = st;
    a.sh = sh;
    a.H = H;
    a.t0 = t0;
    a.n_new = n_new;
    a.t_cap = t_cap;
    a.pg = pg;
    a.rec_stride = 0;
    a.records = records;
    a.mean_q = mean_q;
    a.mean_scale = mean_scale;
    a.status = status;
    a.rotate = 1;
    const size_t smem = sizeof(double) * DQ_MAX_LEVELS + sizeof(int32_t) * DQ_MAX_LEVELS +
                        sizeof(float) * kLambdaSteps + sizeof(int64_t) * kEncStreams +
                        2 * sizeof(uint16_t) * kEncStreams + sizeof(int32_t) * kEncStreams +
                        sizeof(uint4) * DQ_MAX_LEVELS +
                        (size_t)kEncStreams * n + (size_t)kEncStreams * record_bytes;
    dim3 grid((n_new + kEncStreams - 1) / kEncStreams, H, B);
    switch (vpl) {
        case 1: encode_kernel<1, 0, false, true><<<grid, kEncThreads, smem, stream>>>(a); break;
        case 2: encode_kernel<2, 0, false, true><<<grid, kEncThreads, smem, stream>>>(a); break;
        default: encode_kernel<4, 0, false, true><<<grid, kEncThreads, smem, stream>>>(a); break;
    }
    return hip_check("encode_fixed launch", hipGetLastError());
}

}  // namespace dq
