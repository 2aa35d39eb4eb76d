// The HCMS time model (Sec. 3.7 and the appendix's time-model, optimal-chunk
// and speedup equations), host only.
//
//   T_base      = T_0 + T_comm + T_attn
//   T_hcms(C)   = T_0 + T_comm / C + T_attn + C * beta
//   C*          = sqrt(T_comm / beta)
//   S(C)        = 1 / (1 - rho (C - 1) / C + C beta / T_total),  rho = T_comm / T_total
//
// plus a least-squares fit of T(C) = a + b / C + beta C to measured step times,
// which gives a = T_0 + T_attn, b = T_comm and beta for a configuration from a
// sweep over the chunk count.
#include <cmath>

#include "hcms.h"
#include "hcms_internal.h"

namespace {

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

double model_time(double t0, double t_comm, double t_attn, double beta, int C) {
    return t0 + t_comm / C + t_attn + C * beta;
}

// Solves the 3 x 3 system m x = r by Gaussian elimination with partial
// pivoting; false if it is singular.
bool solve3(double m[3][3], double r[3], double x[3]) {
    int p[3] = {0, 1, 2};
    for (int col = 0; col < 3; ++col) {
        int best = col;
        for (int row = col + 1; row < 3; ++row)
            if (std::fabs(m[p[row]][col]) > std::fabs(m[p[best]][col])) best = row;
        const int t = p[col];
        p[col] = p[best];
        p[best] = t;
        const double piv = m[p[col]][col];
        if (!(std::fabs(piv) > 1e-300)) return false;
        for (int row = col + 1; row < 3; ++row) {
            const double f = m[p[row]][col] / piv;
            for (int k = col; k < 3; ++k) m[p[row]][k] -= f * m[p[col]][k];
            r[p[row]] -= f * r[p[col]];
        }
    }
    for (int col = 2; col >= 0; --col) {
        double acc = r[p[col]];
        for (int k = col + 1; k < 3; ++k) acc -= m[p[col]][k] * x[k];
        x[col] = acc / m[p[col]][col];
    }
    return std::isfinite(x[0]) && std::isfinite(x[1]) && std::isfinite(x[2]);
}

}  // namespace

extern "C" {

int hcms_model_time(double t0, double t_comm, double t_attn, double beta, int n_chunks,
                    double *t_out) {
    if (!t_out) return hcms::fail(HCMS_ERR_NULL, "t_out is NULL");
    if (n_chunks < 1) return hcms::fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be >= 1", n_chunks);
    if (!finite_nonneg(t0) || !finite_nonneg(t_comm) || !finite_nonneg(t_attn) || !finite_nonneg(beta))
        return hcms::fail(HCMS_ERR_ARG, "times must be finite and >= 0");
    *t_out = model_time(t0, t_comm, t_attn, beta, n_chunks);
    return hcms::ok();
}

int hcms_model_optimal_chunks(double t_comm, double beta, int H, double *c_real_out) {
    if (H < 1) return hcms::fail(HCMS_ERR_SHAPE, "H=%d must be >= 1", H);
    if (!finite_nonneg(t_comm) || !finite_nonneg(beta))
        return hcms::fail(HCMS_ERR_ARG, "times must be finite and >= 0");
    const double c_real = beta > 0.0 ? std::sqrt(t_comm / beta) : INFINITY;
    if (c_real_out) *c_real_out = c_real;
    // T(C) - const = t_comm / C + C beta is convex in C: the best integer is
    // one of the two around C*, clamped to [1, H]; ties go to fewer chunks.
    int lo = 1, hi = H;
    if (std::isfinite(c_real)) {
        const double f = std::floor(c_real);
        lo = f < 1.0 ? 1 : (f > H ? H : static_cast<int>(f));
        hi = lo < H ? lo + 1 : H;
    } else {
        lo = hi = H;
    }
    const double t_lo = model_time(0.0, t_comm, 0.0, beta, lo);
    const double t_hi = model_time(0.0, t_comm, 0.0, beta, hi);
    hcms::ok();
    return t_hi < t_lo ? hi : lo;
}

int hcms_model_speedup(double rho, double beta_over_total, int n_chunks, double *s_out) {
    if (!s_out) return hcms::fail(HCMS_ERR_NULL, "s_out is NULL");
    if (n_chunks < 1) return hcms::fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be >= 1", n_chunks);
    if (!(rho >= 0.0 && rho <= 1.0) || !finite_nonneg(beta_over_total))
        return hcms::fail(HCMS_ERR_ARG, "rho must be in [0, 1] and beta / T_total >= 0");
    const double C = n_chunks;
    const double denom = 1.0 - rho * (C - 1.0) / C + C * beta_over_total;
    if (!(denom > 0.0)) return hcms::fail(HCMS_ERR_ARG, "the model's time is not positive");
    *s_out = 1.0 / denom;
    return hcms::ok();
}

int hcms_model_fit(const int *chunk_counts, const double *times, int n, double *a_out,
                   double *t_comm_out, double *beta_out) {
    if (!chunk_counts || !times || !a_out || !t_comm_out || !beta_out)
        return hcms::fail(HCMS_ERR_NULL, "an argument is NULL");
    if (n < 3) return hcms::fail(HCMS_ERR_ARG, "need at least 3 points, got %d", n);
    // Normal equations of min sum_i (a + b / C_i + beta C_i - T_i)^2.
    double m[3][3] = {{0}}, r[3] = {0};
    for (int i = 0; i < n; ++i) {
        if (chunk_counts[i] < 1) return hcms::fail(HCMS_ERR_CHUNKS, "chunk count %d < 1", chunk_counts[i]);
        if (!std::isfinite(times[i])) return hcms::fail(HCMS_ERR_ARG, "time %d is not finite", i);
        const double f[3] = {1.0, 1.0 / chunk_counts[i], static_cast<double>(chunk_counts[i])};
        for (int j = 0; j < 3; ++j) {
            r[j] += f[j] * times[i];
            for (int k = 0; k < 3; ++k) m[j][k] += f[j] * f[k];
        }
    }
    double x[3];
    if (!solve3(m, r, x))
        return hcms::fail(HCMS_ERR_ARG, "the fit is singular (fewer than 3 distinct chunk counts)");
    *a_out = x[0];
    *t_comm_out = x[1];
    *beta_out = x[2];
    return hcms::ok();
}

}  // extern "C"
