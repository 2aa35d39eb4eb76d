// The HCMS time model (Sec. 3.7 and the appendix's time-model, optimal-chunk
// and speedup equations), host only.
//
//   T_base      = T_0 + T_comm + T_attn
//   T_hcms(C)   = T_0 + T_comm / C + T_attn + C * beta
//   C*          = sqrt(T_comm / beta)
//   S(C)        = 1 / (1 - rho (C - 1) / C + C beta / T_total),  rho = T_comm / T_total
//
// plus a least-squares fit of T(C) = a + b / C + beta C to measured step times,
// which gives a = T_0 + T_comm and beta for a configuration from a sweep over
// the chunk count.
//
// On one GPU the attention time itself depends on the chunking (the paper's
// model holds it constant): a launch of W workgroups on n slots runs
// floor(W / n) full rounds and, when n does not divide W, one partial round
// that keeps a fraction f = (W mod n) / n of the slots busy.  The chip's
// clock rises when part of it idles, so a partial round takes
// t_round (g0 + (1 - g0) f) rather than a whole t_round.  Summed over the
// launches, T_attn = t_round (sum W / n) + t_round g0 (R - sum W / n) with
// R = sum ceil(W / n) the round count: only the idle share of the partial
// rounds depends on C.  A launch that splits its last round's tiles by key
// segments (attention_split_ways) shortens that round to a third or two
// thirds.  Each launch also drains: its last workgroups finish at different
// times (the XCDs run at different clocks), a cost of `drain` rounds per
// launch on the critical path.  hcms_model_plan_time adds the copies each plan
// leaves on the critical path and its synchronisations; hcms_choose_chunks
// picks the chunk count whose plan (the one HCMS_MODE_AUTO runs) the model
// predicts fastest.
#include <algorithm>
#include <cmath>
#include <vector>

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

// Duration of one launch of W workgroups on n slots, in units of a full round,
// when its last round's tiles are split `ways` ways by key segments (1: not
// split; 2: the round lasts two thirds as long with 2 rem workgroups busy;
// 3: a third as long with 3 rem busy).
double launch_rounds(int64_t W, int64_t n, double g0, int ways) {
    if (W <= 0) return 0.0;
    const int64_t full = W / n, rem = W % n;
    if (rem == 0) return static_cast<double>(full);
    const double f = static_cast<double>(rem * ways) / static_cast<double>(n);
    const double len = ways == 3 ? 1.0 / 3.0 : ways == 2 ? 2.0 / 3.0 : 1.0;
    return static_cast<double>(full) + len * (g0 + (1.0 - g0) * f);
}

bool plan_mode(int m) {
    return m == HCMS_MODE_SERIAL || m == HCMS_MODE_PIPELINED || m == HCMS_MODE_INLINE ||
           m == HCMS_MODE_LANES || m == HCMS_MODE_SLOTS || m == HCMS_MODE_FUSED;
}

// Model time of one plan; arguments already validated.
double plan_time(int S, int d, int dtype, const int *sizes, int C, int mode, int n_cu,
                 double t_round, double g0, double drain, double t_copy, double beta) {
    const int64_t br = hcms::attention_queries_per_block(d);
    const int64_t n = static_cast<int64_t>(n_cu) * hcms::attention_blocks_per_cu(d);
    const int64_t tiles = (static_cast<int64_t>(S) + br - 1) / br;
    int64_t H = 0, total = 0;
    for (int c = 0; c < C; ++c) {
        H += sizes[c];
        total += tiles * sizes[c];
    }
    if (C == 1) mode = HCMS_MODE_SERIAL;
    double attn = 0.0;
    if (mode == HCMS_MODE_LANES) {   // the chunks' workgroups pooled; the remainder past the
                                     // last whole pooled round split by the lanes' last launches
        attn = launch_rounds(total, n, g0, hcms::attention_split_ways(total, S, d, dtype, n_cu)) +
               drain * ((C + 1) / 2);
    } else {
        attn = drain * C;
        for (int c = 0; c < C; ++c) {
            const int64_t W = tiles * sizes[c];
            attn += launch_rounds(W, n, g0, hcms::attention_split_ways(W, S, d, dtype, n_cu));
        }
    }
    attn *= t_round;
    // Copies on the critical path, in head-tensors (a pack moves 3 per head,
    // an unpack 1): all of them when serial; otherwise chunk 0's pack and the
    // last chunk's unpack, plus, in the fused plan, the copies of launches
    // whose last round leaves too few slots idle to carry them.
    double copies;
    if (mode == HCMS_MODE_SERIAL) {
        copies = 4.0 * static_cast<double>(H);
    } else {
        copies = 3.0 * sizes[0] + sizes[C - 1];
        if (mode == HCMS_MODE_FUSED)
            for (int c = 0; c < C; ++c) {
                const int64_t W = tiles * sizes[c];
                const int64_t rem = W % n;
                const int64_t W_run = W - rem + rem * hcms::attention_split_ways(W, S, d, dtype, n_cu);
                const int64_t idle = (n - W_run % n) % n;
                if (idle >= std::max<int64_t>(1, n / 8)) continue;
                if (c + 1 < C) copies += 3.0 * sizes[c + 1];
                if (c >= 1) copies += sizes[c - 1];
            }
    }
    int syncs = 0;
    if (mode == HCMS_MODE_INLINE || mode == HCMS_MODE_LANES) syncs = 4;
    if (mode == HCMS_MODE_PIPELINED || mode == HCMS_MODE_SLOTS) syncs = 2 * C + 3;
    return attn + copies * t_copy + syncs * beta;
}

int check_one_gpu(int S, int d, int dtype, int n_cu, double t_round, double g0, double drain,
                  double t_copy, double beta) {
    if (S < 0) return hcms::fail(HCMS_ERR_SHAPE, "S=%d must be >= 0", S);
    if (d != 64 && d != 128) return hcms::fail(HCMS_ERR_SHAPE, "d=%d must be 64 or 128", d);
    if (dtype != HCMS_BF16 && dtype != HCMS_FP32) return hcms::fail(HCMS_ERR_DTYPE, "dtype %d", dtype);
    if (n_cu < 1) return hcms::fail(HCMS_ERR_ARG, "n_cu=%d must be >= 1", n_cu);
    if (!finite_nonneg(t_round) || !finite_nonneg(t_copy) || !finite_nonneg(beta) ||
        !finite_nonneg(drain))
        return hcms::fail(HCMS_ERR_ARG, "times must be finite and >= 0");
    if (!(g0 > 0.0 && g0 <= 1.0)) return hcms::fail(HCMS_ERR_ARG, "g0=%g must be in (0, 1]", g0);
    return HCMS_OK;
}

}  // namespace

extern "C" {

int hcms_model_plan_time(int S, int d, int dtype, const int *chunk_sizes, int n_chunks, int mode,
                         int n_cu, double t_round, double g0, double drain, double t_copy,
                         double beta, double *t_out) {
    int st;
    if (!t_out || !chunk_sizes) return hcms::fail(HCMS_ERR_NULL, "an argument is NULL");
    if ((st = check_one_gpu(S, d, dtype, n_cu, t_round, g0, drain, t_copy, beta)) != HCMS_OK)
        return st;
    if (n_chunks < 1) return hcms::fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be >= 1", n_chunks);
    for (int c = 0; c < n_chunks; ++c)
        if (chunk_sizes[c] < 1) return hcms::fail(HCMS_ERR_CHUNKS, "chunk %d has %d heads", c, chunk_sizes[c]);
    if (mode == HCMS_MODE_AUTO) {
        int64_t H = 0;
        for (int c = 0; c < n_chunks; ++c) H += chunk_sizes[c];
        if (H > 0x7fffffff) return hcms::fail(HCMS_ERR_CHUNKS, "too many heads");
        mode = hcms::auto_plan(S, d, dtype, chunk_sizes, n_chunks, n_cu);
    }
    if (!plan_mode(mode)) return hcms::fail(HCMS_ERR_ARG, "mode %d is not a plan", mode);
    *t_out = plan_time(S, d, dtype, chunk_sizes, n_chunks, mode, n_cu, t_round, g0, drain, t_copy,
                       beta);
    return hcms::ok();
}

int hcms_choose_chunks(int S, int H, int d, int dtype, int n_cu, double t_round, double g0,
                       double drain, double t_copy, double beta, int max_chunks, int *sizes_out,
                       int *mode_out, double *t_out) {
    int st;
    if (!sizes_out) return hcms::fail(HCMS_ERR_NULL, "sizes_out is NULL");
    if ((st = check_one_gpu(S, d, dtype, n_cu, t_round, g0, drain, t_copy, beta)) != HCMS_OK)
        return st;
    if (H < 1) return hcms::fail(HCMS_ERR_SHAPE, "H=%d must be >= 1", H);
    if (max_chunks < 1) return hcms::fail(HCMS_ERR_CHUNKS, "max_chunks=%d must be >= 1", max_chunks);
    const int top = std::min(H, max_chunks);
    std::vector<int> sizes(top), best_sizes;
    double best_t = INFINITY;
    int best_mode = HCMS_MODE_SERIAL;
    for (int C = 1; C <= top; ++C) {
        for (int c = 0; c < C; ++c) sizes[c] = H / C + (c < H % C ? 1 : 0);
        const int mode = hcms::auto_plan(S, d, dtype, sizes.data(), C, n_cu);
        const double t = plan_time(S, d, dtype, sizes.data(), C, mode, n_cu, t_round, g0, drain,
                                   t_copy, beta);
        if (t < best_t) {   // ties keep the smaller chunk count
            best_t = t;
            best_mode = mode;
            best_sizes.assign(sizes.begin(), sizes.begin() + C);
        }
    }
    std::copy(best_sizes.begin(), best_sizes.end(), sizes_out);
    if (mode_out) *mode_out = best_mode;
    if (t_out) *t_out = best_t;
    hcms::ok();
    return static_cast<int>(best_sizes.size());
}

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
