// Host side of the library: the calibration-free entropy model, argument
// validation and the exported C entry points.
//
// The table build follows Sec. 4.2 (probability model from Gaussian order
// statistics: the min and max of n standard normals are taken at -a_n and
// +a_n, a_n = E[max]), Sec. 4.4 (sharpening p^alpha) and Eq. (rans)
// (integer frequencies summing to 2^p), with the costs of Alg. 1 held as Q16
// integers so the budget test is exact.
#include <algorithm>
#include <cstdio>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "dq_internal.h"

namespace {

thread_local char g_last_error[256] = "";

}  // namespace

int dq::hip_fail(const char* where, hipError_t err) {
    std::snprintf(g_last_error, sizeof(g_last_error), "%s: %s (%s)", where, hipGetErrorName(err),
                  hipGetErrorString(err));
    return DQ_ERR_HIP;
}

namespace {

// Gauss-Legendre nodes and weights on [-1, 1] by Newton iteration on P_k.
void gauss_legendre(int k, std::vector<double>& x, std::vector<double>& w) {
    x.assign(k, 0.0);
    w.assign(k, 0.0);
    for (int i = 0; i < k; ++i) {
        double z = std::cos(M_PI * (i + 0.75) / (k + 0.5));
        double dp = 0.0;
        for (int it = 0; it < 100; ++it) {
            double p0 = 1.0, p1 = z;
            for (int j = 2; j <= k; ++j) {
                double p2 = ((2.0 * j - 1.0) * z * p1 - (j - 1.0) * p0) / j;
                p0 = p1;
                p1 = p2;
            }
            dp = k * (z * p1 - p0) / (z * z - 1.0);
            double dz = p1 / dp;
            z -= dz;
            if (std::fabs(dz) < 1e-16) break;
        }
        x[i] = z;
        w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
    }
}

double normal_cdf(double x) { return 0.5 * std::erfc(-x / std::sqrt(2.0)); }

// a_n = integral of x n phi(x) Phi(x)^(n-1) dx, composite 12-point
// Gauss-Legendre over [-14, 14] in panels of 0.02.
double expected_max(int n) {
    if (n <= 1) return 0.0;
    std::vector<double> gx, gw;
    gauss_legendre(12, gx, gw);
    const double lo = -14.0, h = 0.02;
    const int panels = 1400;
    const double inv_sqrt_2pi = 1.0 / std::sqrt(2.0 * M_PI);
    double total = 0.0;
    for (int k = 0; k < panels; ++k) {
        double a = lo + k * h, mid = a + 0.5 * h, part = 0.0;
        for (size_t i = 0; i < gx.size(); ++i) {
            double x = mid + 0.5 * h * gx[i];
            double f = x * n * inv_sqrt_2pi * std::exp(-0.5 * x * x) *
                       std::pow(normal_cdf(x), (double)(n - 1));
            part += gw[i] * f;
        }
        total += 0.5 * h * part;
    }
    return total;
}

struct Built {
    dq_table_info info;
    int32_t freq[DQ_MAX_LEVELS];
    int32_t cum[DQ_MAX_LEVELS];
    int32_t cost[DQ_MAX_LEVELS];
    float lam[dq::kLambdaSteps];
};

int validate(const dq_config* c) {
    if (!c) return DQ_ERR_INVALID_ARG;
    const int n = c->head_dim;
    if (n < 64 || n > 1024 || (n & (n - 1))) return DQ_ERR_INVALID_ARG;
    if (c->levels < 2 || c->levels > DQ_MAX_LEVELS) return DQ_ERR_INVALID_ARG;
    if (c->precision_bits < 8 || c->precision_bits > 12) return DQ_ERR_INVALID_ARG;
    if (c->record_bytes < 9 || c->record_bytes > 2 * n + 8) return DQ_ERR_INVALID_ARG;
    if (!(c->alpha >= 1.0) || !(c->alpha <= 64.0)) return DQ_ERR_INVALID_ARG;
    if ((c->levels / 2) > (1 << (c->precision_bits - 1))) return DQ_ERR_INVALID_ARG;
    if (c->prerotated != 0 && c->prerotated != 1) return DQ_ERR_INVALID_ARG;
    return DQ_OK;
}

int build(const dq_config* c, Built* out) {
    const int n = c->head_dim, M = c->levels, p = c->precision_bits;
    const int64_t total = int64_t(1) << p;
    const int half = M / 2;
    const double a = expected_max(n);

    // Level masses: lower half by CDF differences, centre by erf, mirrored.
    double q[DQ_MAX_LEVELS];
    double prev = 0.0;
    for (int m = 0; m < half; ++m) {
        double edge = a * ((2.0 * (m + 1) - 1.0) / (M - 1) - 1.0);
        double cur = normal_cdf(edge);
        q[m] = cur - prev;
        prev = cur;
    }
    if (M % 2) q[half] = std::erf(a / (M - 1) / std::sqrt(2.0));
    for (int m = 0; m < half; ++m) q[M - 1 - m] = q[m];

    // Sharpening.
    double w[DQ_MAX_LEVELS], wsum = 0.0;
    for (int m = 0; m < M; ++m) {
        w[m] = std::pow(q[m], c->alpha);
        wsum += w[m];
    }

    // Symmetric largest-remainder apportionment of the lower half.
    double g[DQ_MAX_LEVELS];
    double gsum = 0.0;
    for (int m = 0; m < half; ++m) {
        g[m] = (w[m] / wsum) * (double)total;
        gsum += g[m];
    }
    int64_t H;
    if (M % 2) {
        H = (int64_t)std::floor(gsum + 0.5);
        H = std::min<int64_t>(H, (total - 1) / 2);
    } else {
        H = total / 2;
    }
    if (H < half) return DQ_ERR_INVALID_ARG;
    int64_t f[DQ_MAX_LEVELS];
    int64_t fsum = 0;
    for (int m = 0; m < half; ++m) {
        f[m] = std::max<int64_t>(1, (int64_t)std::floor(g[m]));
        fsum += f[m];
    }
    int64_t deficit = H - fsum;
    if (deficit > 0) {
        std::vector<int> order(half);
        for (int m = 0; m < half; ++m) order[m] = m;
        std::stable_sort(order.begin(), order.end(), [&](int i, int j) {
            double fi = g[i] - std::floor(g[i]), fj = g[j] - std::floor(g[j]);
            return fi > fj;
        });
        for (int64_t k = 0; deficit > 0; ++k, --deficit) f[order[k % half]] += 1;
    }
    while (deficit < 0) {
        int best = 0;
        for (int m = 1; m < half; ++m)
            if (f[m] > f[best]) best = m;
        if (f[best] <= 1) return DQ_ERR_INVALID_ARG;
        f[best] -= 1;
        ++deficit;
    }
    int64_t full[DQ_MAX_LEVELS];
    for (int m = 0; m < half; ++m) {
        full[m] = f[m];
        full[M - 1 - m] = f[m];
    }
    if (M % 2) full[half] = total - 2 * H;

    std::memset(out, 0, sizeof(*out));
    int64_t run = 0;
    int32_t rmin = INT32_MAX, cheapest = 0;
    for (int m = 0; m < M; ++m) {
        out->freq[m] = (int32_t)full[m];
        out->cum[m] = (int32_t)run;
        run += full[m];
        double r = (double)p - std::log2((double)full[m]);
        out->cost[m] = (int32_t)std::floor(r * 65536.0 + 0.5);
        if (out->cost[m] < rmin) {
            rmin = out->cost[m];
            cheapest = m;
        }
    }
    if (run != total) return DQ_ERR_INVALID_ARG;
    for (int k = 0; k < dq::kLambdaSteps; ++k)
        out->lam[k] = (float)std::exp2((double)k / dq::kLambdaSteps);

    dq_table_info& info = out->info;
    info.record_bytes = c->record_bytes;
    info.budget_q16 = (int64_t)(8 * (c->record_bytes - 4) - 32) * 65536;
    info.min_cost_q16 = (int64_t)n * rmin;
    info.cheapest = cheapest;
    info.expected_max = a;
    info.feasible = (info.budget_q16 > 0 && info.min_cost_q16 <= info.budget_q16) ? 1 : 0;
    return info.feasible ? DQ_OK : DQ_ERR_INFEASIBLE;
}

bool table_args_ok(const dq_tables* t) { return t && t->dev_block; }

}  // namespace

extern "C" {

int dq_compute_tables(const dq_config* cfg, dq_table_info* info, int32_t* freq, int32_t* cum,
                      int32_t* cost_q16, uint8_t* sym_of_z, float* lambda512) {
    int rc = validate(cfg);
    if (rc != DQ_OK) return rc;
    Built b;
    rc = build(cfg, &b);
    if (rc != DQ_OK && rc != DQ_ERR_INFEASIBLE) return rc;
    const int M = cfg->levels;
    if (info) *info = b.info;
    if (freq) std::memcpy(freq, b.freq, sizeof(int32_t) * M);
    if (cum) std::memcpy(cum, b.cum, sizeof(int32_t) * M);
    if (cost_q16) std::memcpy(cost_q16, b.cost, sizeof(int32_t) * M);
    if (lambda512) std::memcpy(lambda512, b.lam, sizeof(float) * dq::kLambdaSteps);
    if (sym_of_z) {
        for (int m = 0; m < M; ++m)
            for (int z = b.cum[m]; z < b.cum[m] + b.freq[m]; ++z) sym_of_z[z] = (uint8_t)m;
    }
    return rc;
}

int dq_build_tables(const dq_config* cfg, dq_tables** out, dq_table_info* info) {
    if (!out) return DQ_ERR_INVALID_ARG;
    *out = nullptr;
    int rc = validate(cfg);
    if (rc != DQ_OK) return rc;
    Built b;
    rc = build(cfg, &b);
    if (info) *info = b.info;
    if (rc != DQ_OK) return rc;

    const int M = cfg->levels, P = 1 << cfg->precision_bits;
    // device block: lut64[P] | lut[P] u32 | freq[64] | cum[64] | cost[64] | lam[512]
    const size_t lut64_bytes = sizeof(uint32_t) * 2 * P;
    const size_t lut_bytes = lut64_bytes + sizeof(uint32_t) * P;
    const size_t small = sizeof(int32_t) * DQ_MAX_LEVELS;
    const size_t bytes = lut_bytes + 3 * small + sizeof(float) * dq::kLambdaSteps;
    std::vector<uint8_t> host(bytes, 0);
    uint32_t* lut64 = reinterpret_cast<uint32_t*>(host.data());
    uint32_t* lut = reinterpret_cast<uint32_t*>(host.data() + lut64_bytes);
    for (int m = 0; m < M; ++m)
        for (int z = b.cum[m]; z < b.cum[m] + b.freq[m]; ++z) {
            lut[z] = (uint32_t)(z - b.cum[m]) | ((uint32_t)b.freq[m] << 12) | ((uint32_t)m << 24);
            lut64[2 * z] = 8u * (uint32_t)b.freq[m] | ((uint32_t)m << 24);
            lut64[2 * z + 1] = 8u * (uint32_t)(z - b.cum[m]);
        }
    std::memcpy(host.data() + lut_bytes, b.freq, sizeof(int32_t) * M);
    std::memcpy(host.data() + lut_bytes + small, b.cum, sizeof(int32_t) * M);
    std::memcpy(host.data() + lut_bytes + 2 * small, b.cost, sizeof(int32_t) * M);
    std::memcpy(host.data() + lut_bytes + 3 * small, b.lam, sizeof(float) * dq::kLambdaSteps);

    dq_tables* t = new (std::nothrow) dq_tables;
    if (!t) return DQ_ERR_INVALID_ARG;
    std::memset(t, 0, sizeof(*t));
    t->cfg = *cfg;
    t->info = b.info;
    std::memcpy(t->freq, b.freq, sizeof(t->freq));
    std::memcpy(t->cum, b.cum, sizeof(t->cum));
    std::memcpy(t->cost, b.cost, sizeof(t->cost));
    if ((rc = dq::hip_check("hipGetDevice", hipGetDevice(&t->device))) != DQ_OK) {
        delete t;
        return rc;
    }
    if ((rc = dq::hip_check("hipMalloc", hipMalloc(&t->dev_block, bytes))) != DQ_OK) {
        delete t;
        return rc;
    }
    rc = dq::hip_check("hipMemcpy", hipMemcpy(t->dev_block, host.data(), bytes, hipMemcpyHostToDevice));
    if (rc != DQ_OK) {
        (void)hipFree(t->dev_block);
        delete t;
        return rc;
    }
    uint8_t* base = static_cast<uint8_t*>(t->dev_block);
    t->dev.lut64 = reinterpret_cast<const uint2*>(base);
    t->dev.lut = reinterpret_cast<const uint32_t*>(base + lut64_bytes);
    t->dev.freq = reinterpret_cast<const int32_t*>(base + lut_bytes);
    t->dev.cum = reinterpret_cast<const int32_t*>(base + lut_bytes + small);
    t->dev.cost = reinterpret_cast<const int32_t*>(base + lut_bytes + 2 * small);
    t->dev.lam = reinterpret_cast<const float*>(base + lut_bytes + 3 * small);
    *out = t;
    return DQ_OK;
}

void dq_free_tables(dq_tables* t) {
    if (!t) return;
    if (t->dev_block) (void)hipFree(t->dev_block);
    delete t;
}

// token_stride > 0: per-token streams over the H heads (the table's n must be
// 128 H), records at that stride; 0: per (token, head) streams.
static int encode_kv(const dq_tables* t, const dq::Pages& pg, const uint16_t* kv, int64_t sb, int64_t st,
                     int64_t sh, int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                     uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status, void* stream,
                     int32_t token_stride = 0) {
    if (!table_args_ok(t) || !kv || !records) return DQ_ERR_INVALID_ARG;
    if (token_stride > 0) {
        if ((H != 1 && H != 2 && H != 4 && H != 8) || t->cfg.head_dim != 128 * H) return DQ_ERR_INVALID_ARG;
    } else if (t->cfg.head_dim > 256) {
        return DQ_ERR_INVALID_ARG;
    }
    if (B < 0 || H <= 0 || t0 < 0 || n_new < 0 || t_cap <= 0 || t0 + n_new > t_cap)
        return DQ_ERR_INVALID_ARG;
    if (B > 65535 || H > 65535) return DQ_ERR_INVALID_ARG;   // grid dimensions
    if (sb < 0 || st < 0 || sh < 0) return DQ_ERR_INVALID_ARG;
    const bool keys = mean_q != nullptr;
    if (keys != (mean_scale != nullptr)) return DQ_ERR_INVALID_ARG;
    if (keys && ((t0 % DQ_MEAN_WINDOW) || (n_new % DQ_MEAN_WINDOW) || (t_cap % DQ_MEAN_WINDOW)))
        return DQ_ERR_INVALID_ARG;
    if (B == 0 || n_new == 0) return DQ_OK;
    return dq::launch_encode(t, pg, kv, sb, st, sh, B, H, t0, n_new, t_cap, records, mean_q,
                             mean_scale, status, static_cast<hipStream_t>(stream), token_stride);
}

static const dq::Pages kContiguous{nullptr, 0, 0, 0};

// A paged layout: page length a power of two in [128, 2^20], a logical
// capacity max_pages * page_tokens within int32.
static int paging(const int32_t* bt, int32_t max_pages, int32_t page_tokens, int32_t num_pages,
                  dq::Pages* pg, int32_t* t_cap) {
    if (!bt || max_pages <= 0 || num_pages <= 0) return DQ_ERR_INVALID_ARG;
    if (page_tokens < DQ_MEAN_WINDOW || page_tokens > (1 << 20) || (page_tokens & (page_tokens - 1)))
        return DQ_ERR_INVALID_ARG;
    if ((int64_t)max_pages * page_tokens > 0x7FFFFFFF) return DQ_ERR_INVALID_ARG;
    int shift = 0;
    while ((1 << shift) < page_tokens) ++shift;
    *pg = dq::Pages{bt, max_pages, shift, num_pages};
    *t_cap = max_pages * page_tokens;
    return DQ_OK;
}

int dq_encode_kv(const dq_tables* t, const uint16_t* kv, int64_t sb, int64_t st, int64_t sh,
                 int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                 uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status,
                 void* stream) {
    return encode_kv(t, kContiguous, kv, sb, st, sh, B, H, t0, n_new, t_cap, records, mean_q, mean_scale,
                     status, stream);
}

int dq_encode_kv_paged(const dq_tables* t, const uint16_t* kv, int64_t sb, int64_t st, int64_t sh,
                       int32_t B, int32_t H, int32_t t0, int32_t n_new, const int32_t* block_table,
                       int32_t max_pages, int32_t page_tokens, int32_t num_pages, uint8_t* record_pool,
                       int8_t* mean_q_pool, uint16_t* mean_scale_pool, uint32_t* status, void* stream) {
    dq::Pages pg;
    int32_t t_cap = 0;
    if (int rc = paging(block_table, max_pages, page_tokens, num_pages, &pg, &t_cap)) return rc;
    return encode_kv(t, pg, kv, sb, st, sh, B, H, t0, n_new, t_cap, record_pool, mean_q_pool, mean_scale_pool,
                     status, stream);
}

int32_t dq_token_record_stride(const dq_tables* t) {
    if (!table_args_ok(t)) return 0;
    return (t->cfg.record_bytes + 15) & ~15;
}

int dq_encode_kv_token(const dq_tables* t, const uint16_t* kv, int64_t sb, int64_t st, int64_t sh,
                       int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                       uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status,
                       void* stream) {
    const int32_t stride = dq_token_record_stride(t);
    if (stride <= 0) return DQ_ERR_INVALID_ARG;
    return encode_kv(t, kContiguous, kv, sb, st, sh, B, H, t0, n_new, t_cap, records, mean_q, mean_scale,
                     status, stream, stride);
}

int dq_encode_kv_token_paged(const dq_tables* t, const uint16_t* kv, int64_t sb, int64_t st, int64_t sh,
                             int32_t B, int32_t H, int32_t t0, int32_t n_new, const int32_t* block_table,
                             int32_t max_pages, int32_t page_tokens, int32_t num_pages, uint8_t* record_pool,
                             int8_t* mean_q_pool, uint16_t* mean_scale_pool, uint32_t* status, void* stream) {
    const int32_t stride = dq_token_record_stride(t);
    if (stride <= 0) return DQ_ERR_INVALID_ARG;
    dq::Pages pg;
    int32_t t_cap = 0;
    if (int rc = paging(block_table, max_pages, page_tokens, num_pages, &pg, &t_cap)) return rc;
    return encode_kv(t, pg, kv, sb, st, sh, B, H, t0, n_new, t_cap, record_pool, mean_q_pool, mean_scale_pool,
                     status, stream, stride);
}

int32_t dq_fixed_bits(int32_t head_dim, int32_t record_bytes) {
    if (head_dim <= 0 || record_bytes <= 4) return 0;
    const int64_t b = 8 * (int64_t)(record_bytes - 4) / head_dim;
    return b >= 1 && b <= 8 ? (int32_t)b : 0;
}

int dq_encode_kv_fixed(int32_t head_dim, int32_t record_bytes, const uint16_t* kv, int64_t sb, int64_t st,
                       int64_t sh, int32_t B, int32_t H, int32_t t0, int32_t n_new, int32_t t_cap,
                       uint8_t* records, int8_t* mean_q, uint16_t* mean_scale, uint32_t* status, void* stream) {
    if (!kv || !records) return DQ_ERR_INVALID_ARG;
    if (head_dim != 64 && head_dim != 128 && head_dim != 256) return DQ_ERR_INVALID_ARG;
    if (dq_fixed_bits(head_dim, record_bytes) == 0 || record_bytes > 2 * head_dim + 8) return DQ_ERR_INVALID_ARG;
    if (B < 0 || H <= 0 || t0 < 0 || n_new < 0 || t_cap <= 0 || t0 + n_new > t_cap) return DQ_ERR_INVALID_ARG;
    if (B > 65535 || H > 65535) return DQ_ERR_INVALID_ARG;
    if (sb < 0 || st < 0 || sh < 0) return DQ_ERR_INVALID_ARG;
    const bool keys = mean_q != nullptr;
    if (keys != (mean_scale != nullptr)) return DQ_ERR_INVALID_ARG;
    if (keys && ((t0 % DQ_MEAN_WINDOW) || (n_new % DQ_MEAN_WINDOW) || (t_cap % DQ_MEAN_WINDOW)))
        return DQ_ERR_INVALID_ARG;
    if (B == 0 || n_new == 0) return DQ_OK;
    return dq::launch_encode_fixed(head_dim, record_bytes, kContiguous, kv, sb, st, sh, B, H, t0, n_new, t_cap,
                                   records, mean_q, mean_scale, status, static_cast<hipStream_t>(stream));
}

int dq_decode_attention_fixed_partial(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                      const uint8_t* k_records, const int8_t* k_mean_q,
                                      const uint16_t* k_mean_scale, const uint8_t* v_records,
                                      const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                                      size_t ws_bytes, uint32_t* status, void* stream) {
    if (B <= 0 || B > 65535 || Hkv <= 0 || Hkv > 65535 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 4)
        return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW) return DQ_ERR_INVALID_ARG;
    if (!q || !k_records || !k_mean_q || !k_mean_scale || !v_records || !seq_lens) return DQ_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128)) return DQ_ERR_WORKSPACE;
    return dq::launch_attention_fixed_partial(kContiguous, q, B, Hq, Hkv, k_records, k_mean_q, k_mean_scale,
                                              v_records, seq_lens, t_cap, scale, ws, status,
                                              static_cast<hipStream_t>(stream));
}

size_t dq_decode_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t t_cap, int32_t d) {
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || t_cap <= 0 || d <= 0) return 0;
    return dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, d);
}

static int check_attention(const dq_tables* tk, const dq_tables* tv, int32_t B, int32_t Hq,
                           int32_t Hkv, int32_t t_cap) {
    if (!table_args_ok(tk) || !table_args_ok(tv)) return DQ_ERR_INVALID_ARG;
    if (tk->cfg.head_dim != 128 || tv->cfg.head_dim != 128) return DQ_ERR_INVALID_ARG;
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 8) return DQ_ERR_INVALID_ARG;
    if (B > 65535 || Hkv > 65535) return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW) return DQ_ERR_INVALID_ARG;
    return DQ_OK;
}

static int attention_partial(const dq_tables* tk, const dq_tables* tv, const dq::Pages& pg, const uint16_t* q,
                             int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* krec, const int8_t* kmq,
                             const uint16_t* kms, const uint8_t* vrec, const int32_t* seq_lens, int32_t t_cap,
                             float scale, void* ws, size_t ws_bytes, uint32_t* status, void* stream) {
    int rc = check_attention(tk, tv, B, Hq, Hkv, t_cap);
    if (rc != DQ_OK) return rc;
    if (!q || !krec || !kmq || !kms || !vrec || !seq_lens) return DQ_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128))
        return DQ_ERR_WORKSPACE;
    return dq::launch_attention_partial(tk, tv, pg, q, B, Hq, Hkv, krec, kmq, kms, vrec, seq_lens,
                                        t_cap, scale, ws, status,
                                        static_cast<hipStream_t>(stream));
}

int dq_decode_attention_partial(const dq_tables* tk, const dq_tables* tv, const uint16_t* q,
                                int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* krec,
                                const int8_t* kmq, const uint16_t* kms, const uint8_t* vrec,
                                const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                                size_t ws_bytes, uint32_t* status, void* stream) {
    return attention_partial(tk, tv, kContiguous, q, B, Hq, Hkv, krec, kmq, kms, vrec, seq_lens, t_cap, scale,
                             ws, ws_bytes, status, stream);
}

static int token_partial(const dq_tables* tk, const dq_tables* tv, const dq::Pages& pg, const uint16_t* q,
                         int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* k_records, const int8_t* k_mean_q,
                         const uint16_t* k_mean_scale, const uint8_t* v_records, const int32_t* seq_lens,
                         int32_t t_cap, float scale, void* ws, size_t ws_bytes, uint32_t* status, void* stream) {
    if (!table_args_ok(tk) || !table_args_ok(tv)) return DQ_ERR_INVALID_ARG;
    if (Hkv != 1 && Hkv != 2 && Hkv != 4 && Hkv != 8) return DQ_ERR_INVALID_ARG;
    if (tk->cfg.head_dim != 128 * Hkv || tv->cfg.head_dim != 128 * Hkv) return DQ_ERR_INVALID_ARG;
    if (B <= 0 || B > 65535 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 8) return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW) return DQ_ERR_INVALID_ARG;
    if (!q || !k_records || !k_mean_q || !k_mean_scale || !v_records || !seq_lens) return DQ_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128)) return DQ_ERR_WORKSPACE;
    return dq::launch_attention_token_partial(tk, tv, pg, q, B, Hq, Hkv, k_records, dq_token_record_stride(tk),
                                              k_mean_q, k_mean_scale, v_records, dq_token_record_stride(tv),
                                              seq_lens, t_cap, scale, ws, status, static_cast<hipStream_t>(stream));
}

int dq_decode_attention_token_partial(const dq_tables* tk, const dq_tables* tv, const uint16_t* q, int32_t B,
                                      int32_t Hq, int32_t Hkv, const uint8_t* k_records, const int8_t* k_mean_q,
                                      const uint16_t* k_mean_scale, const uint8_t* v_records,
                                      const int32_t* seq_lens, int32_t t_cap, float scale, void* ws,
                                      size_t ws_bytes, uint32_t* status, void* stream) {
    return token_partial(tk, tv, kContiguous, q, B, Hq, Hkv, k_records, k_mean_q, k_mean_scale, v_records,
                         seq_lens, t_cap, scale, ws, ws_bytes, status, stream);
}

int dq_decode_attention_token_paged_partial(const dq_tables* tk, const dq_tables* tv, const uint16_t* q,
                                            int32_t B, int32_t Hq, int32_t Hkv, const uint8_t* k_pool,
                                            const int8_t* mean_q_pool, const uint16_t* mean_scale_pool,
                                            const uint8_t* v_pool, const int32_t* block_table, int32_t max_pages,
                                            int32_t page_tokens, int32_t num_pages, const int32_t* seq_lens,
                                            float scale, void* ws, size_t ws_bytes, uint32_t* status,
                                            void* stream) {
    dq::Pages pg;
    int32_t t_cap = 0;
    if (int rc = paging(block_table, max_pages, page_tokens, num_pages, &pg, &t_cap)) return rc;
    return token_partial(tk, tv, pg, q, B, Hq, Hkv, k_pool, mean_q_pool, mean_scale_pool, v_pool, seq_lens, t_cap,
                         scale, ws, ws_bytes, status, stream);
}

int dq_decode_attention_paged_partial(const dq_tables* tk, const dq_tables* tv, const uint16_t* q, int32_t B,
                                      int32_t Hq, int32_t Hkv, const uint8_t* k_pool, const int8_t* mean_q_pool,
                                      const uint16_t* mean_scale_pool, const uint8_t* v_pool,
                                      const int32_t* block_table, int32_t max_pages, int32_t page_tokens,
                                      int32_t num_pages, const int32_t* seq_lens, float scale, void* ws,
                                      size_t ws_bytes, uint32_t* status, void* stream) {
    dq::Pages pg;
    int32_t t_cap = 0;
    if (int rc = paging(block_table, max_pages, page_tokens, num_pages, &pg, &t_cap)) return rc;
    return attention_partial(tk, tv, pg, q, B, Hq, Hkv, k_pool, mean_q_pool, mean_scale_pool, v_pool, seq_lens,
                             t_cap, scale, ws, ws_bytes, status, stream);
}

int dq_decode_attention_merge(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* seq_lens,
                              int32_t t_cap, const void* ws, size_t ws_bytes, float* out,
                              void* stream) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 8 || B > 65535)
        return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW || !seq_lens || !out) return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128))
        return DQ_ERR_WORKSPACE;
    return dq::launch_attention_merge(B, Hq, Hkv, seq_lens, t_cap, ws, out,
                                      static_cast<hipStream_t>(stream));
}

int dq_decode_attention(const dq_tables* tk, const dq_tables* tv, const uint16_t* q, int32_t B,
                        int32_t Hq, int32_t Hkv, const uint8_t* krec, const int8_t* kmq,
                        const uint16_t* kms, const uint8_t* vrec, const int32_t* seq_lens,
                        int32_t t_cap, float scale, float* out, void* ws, size_t ws_bytes,
                        uint32_t* status, void* stream) {
    if (!out) return DQ_ERR_INVALID_ARG;
    int rc = dq_decode_attention_partial(tk, tv, q, B, Hq, Hkv, krec, kmq, kms, vrec, seq_lens,
                                         t_cap, scale, ws, ws_bytes, status, stream);
    if (rc != DQ_OK) return rc;
    return dq_decode_attention_merge(B, Hq, Hkv, seq_lens, t_cap, ws, ws_bytes, out, stream);
}

int dq_decode_attention_no_alloc(const dq_tables* tk, const dq_tables* tv, const uint16_t* q, int32_t B,
                                 int32_t Hq, int32_t Hkv, const uint8_t* krec, const int8_t* kmq,
                                 const uint16_t* kms, const uint8_t* vrec, const int32_t* seq_lens,
                                 int32_t t_cap, float scale, float* out, uint32_t* status, void* stream) {
    int rc = check_attention(tk, tv, B, Hq, Hkv, t_cap);
    if (rc != DQ_OK) return rc;
    if (!q || !krec || !kmq || !kms || !vrec || !seq_lens || !out) return DQ_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    // the workspace of this call's own chunk plan, packed: header, then
    // accumulators, maxima and sums of B Hq (chunks + 4) slots
    const int64_t slots = dq::attention_plan_slots(B, Hq, Hkv, t_cap);
    const int64_t need = dq::kWsHeader + slots * (128 + 2) * (int64_t)sizeof(float);
    if (need > (int64_t)DQ_NO_ALLOC_SCRATCH_BYTES) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "dq_decode_attention_no_alloc: %lld bytes of split-K workspace needed, the static "
                      "scratch holds %lld",
                      (long long)need, (long long)DQ_NO_ALLOC_SCRATCH_BYTES);
        return DQ_ERR_WORKSPACE;
    }
    void* ws = nullptr;
    if ((rc = dq::no_alloc_scratch(&ws))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = dq::launch_attention_partial(tk, tv, kContiguous, q, B, Hq, Hkv, krec, kmq, kms, vrec, seq_lens, t_cap,
                                      scale, ws, status, s, slots);
    if (rc != DQ_OK) return rc;
    return dq::launch_attention_merge(B, Hq, Hkv, seq_lens, t_cap, ws, out, s, slots);
}

// Shared checks of the residual-window calls (the window kernels read q, the
// key rows and the value rows in 16- and 4-byte pieces).
static int check_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, const uint16_t* res_k,
                          const uint16_t* res_v, const int32_t* seq_lens, const int32_t* res_lens, int32_t r_cap,
                          int32_t t_cap, float scale, const void* ws, size_t ws_bytes) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 8 || B > 65535 || Hkv > 65535)
        return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW || r_cap <= 0 || r_cap > 256) return DQ_ERR_INVALID_ARG;
    if (!q || !res_k || !res_v || !seq_lens || !res_lens || !std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(res_k) | reinterpret_cast<uintptr_t>(res_v) |
         reinterpret_cast<uintptr_t>(q)) & 15)
        return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128)) return DQ_ERR_WORKSPACE;
    return DQ_OK;
}

int dq_decode_attention_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                 const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                                 const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                                 void* ws, size_t ws_bytes, void* stream) {
    const int rc = check_residual(q, B, Hq, Hkv, res_k, res_v, seq_lens, res_lens, r_cap, t_cap, scale, ws,
                                  ws_bytes);
    if (rc != DQ_OK) return rc;
    return dq::launch_attention_residual(q, B, Hq, Hkv, res_k, res_v, seq_lens, res_lens, r_cap, t_cap, scale,
                                         ws, static_cast<hipStream_t>(stream));
}

int dq_decode_attention_merge_residual(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv,
                                       const uint16_t* res_k, const uint16_t* res_v, const int32_t* seq_lens,
                                       const int32_t* res_lens, int32_t r_cap, int32_t t_cap, float scale,
                                       const void* ws, size_t ws_bytes, float* out, void* stream) {
    const int rc = check_residual(q, B, Hq, Hkv, res_k, res_v, seq_lens, res_lens, r_cap, t_cap, scale, ws,
                                  ws_bytes);
    if (rc != DQ_OK) return rc;
    if (!out) return DQ_ERR_INVALID_ARG;
    return dq::launch_attention_merge_residual(q, B, Hq, Hkv, res_k, res_v, seq_lens, res_lens, r_cap, t_cap,
                                               scale, const_cast<void*>(ws), out,
                                               static_cast<hipStream_t>(stream));
}

int dq_bf16_decode_attention_partial(const uint16_t* q, int32_t B, int32_t Hq, int32_t Hkv, const uint16_t* k,
                                     const uint16_t* v, const int32_t* seq_lens, int32_t t_cap, float scale,
                                     void* ws, size_t ws_bytes, void* stream) {
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 8 || B > 65535 || Hkv > 65535)
        return DQ_ERR_INVALID_ARG;
    if (t_cap <= 0 || t_cap % DQ_MEAN_WINDOW) return DQ_ERR_INVALID_ARG;
    if (!q || !k || !v || !seq_lens || !std::isfinite(scale)) return DQ_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15) return DQ_ERR_INVALID_ARG;
    if (!ws || ws_bytes < dq::attention_workspace_bytes(B, Hq, Hkv, t_cap, 128)) return DQ_ERR_WORKSPACE;
    return dq::launch_bf16_partial(q, B, Hq, Hkv, k, v, seq_lens, t_cap, scale, ws,
                                   static_cast<hipStream_t>(stream));
}

int dq_residual_append(const uint16_t* k_new, const uint16_t* v_new, int32_t B, int32_t Hkv, int32_t d,
                       uint16_t* res_k, uint16_t* res_v, const int32_t* seq_lens, int32_t* res_lens,
                       int32_t r_cap, uint32_t* status, void* stream) {
    if (B <= 0 || Hkv <= 0 || d != 128 || r_cap <= 0 || B > 0x7FFFFFFF / 2) return DQ_ERR_INVALID_ARG;
    if (!k_new || !v_new || !res_k || !res_v || !seq_lens || !res_lens) return DQ_ERR_INVALID_ARG;
    return dq::launch_residual_append(k_new, v_new, B, Hkv, res_k, res_v, seq_lens, res_lens, r_cap, status,
                                      static_cast<hipStream_t>(stream));
}

int dq_residual_commit(int32_t* seq_lens, int32_t* res_lens, int32_t B, int32_t n, uint32_t* status,
                       void* stream) {
    if (B <= 0 || n < 0 || !seq_lens || !res_lens) return DQ_ERR_INVALID_ARG;
    if (n == 0) return DQ_OK;
    return dq::launch_residual_commit(seq_lens, res_lens, B, n, status, static_cast<hipStream_t>(stream));
}

int dq_decode_symbols(const dq_tables* t, const uint8_t* records, int64_t n_streams, uint8_t* sym,
                      uint16_t* header, uint32_t* status, void* stream) {
    if (!table_args_ok(t) || n_streams < 0 || (n_streams > 0 && (!records || !sym)))
        return DQ_ERR_INVALID_ARG;
    if (n_streams == 0) return DQ_OK;
    return dq::launch_decode_symbols(t, records, n_streams, sym, header, status,
                                     static_cast<hipStream_t>(stream));
}

const char* dq_last_error(void) { return g_last_error; }

const char* dq_strerror(int code) {
    switch (code) {
        case DQ_OK: return "ok";
        case DQ_ERR_INVALID_ARG: return "invalid argument";
        case DQ_ERR_INFEASIBLE: return "infeasible: n * min cost exceeds the record budget";
        case DQ_ERR_HIP: return "HIP runtime error";
        case DQ_ERR_WORKSPACE: return "workspace missing or too small";
        default: return "unknown error";
    }
}

}  // extern "C"
