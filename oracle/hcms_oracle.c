/*
 * Oracle for the single-GPU share of HCMS (head-chunked multi-stream
 * attention, arXiv 2607.01817).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or calls
 * this file: only the test suite, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no source, header, table or helper with the HIP
 * library; the two are compared on the same seeded inputs.
 *
 * Everything here is deliberately plain: explicit loops, fp64 arithmetic,
 * no tiling, no fusion, no online softmax.
 *
 *   oracle_attention_rows  Sec. 3.3, Property "Computational Independence of
 *                          Multi-Head Attention": the output of one head is a
 *                          function of that head's Q, K, V only.  The function
 *                          f is scaled-dot-product softmax attention (Alg. 1
 *                          names FlashAttention or SDPA as the kernel), over the
 *                          full sequence with no mask (bidirectional video DiT
 *                          attention, Sec. 2.1).  Written as the textbook
 *                          two-pass softmax.
 *   oracle_pack            Sec. 3.3, split of Q/K/V along the head dimension
 *                          into chunk c (heads [h0, h0+Hc)), combined with the
 *                          local share of the input all-to-all of Sec. 3.1
 *                          (sequence-sharded -> head-sharded).  Index formula:
 *                            dst[j][p*(S/P)+s][e] = src[p][s][h0+j][e].
 *   oracle_unpack          The inverse (output all-to-all + concatenation along
 *                          heads, Alg. 1): dst[p][s][h0+j][e] = src[j][p*(S/P)+s][e];
 *                          heads outside the chunk are left untouched.
 *   oracle_attention_backward
 *                          The gradient of that attention with respect to Q, K
 *                          and V for a given output gradient (the training use
 *                          of Sec. 4, correctness and training validation in
 *                          the appendix), written as the chain rule through the
 *                          softmax with full rows, no recomputation tricks.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/*
 * One head, a list of query rows.
 *   q       : [Sq][d] row-major fp64 queries (the exact stored values, widened)
 *   k, v    : [S][d] row-major fp64 keys and values
 *   rows    : n_rows query indices in [0, Sq)
 *   out     : [n_rows][d]
 * For each listed query i:
 *   s_j = scale * sum_t q[i][t] * k[j][t]          for all j < S
 *   m   = max_j s_j
 *   l   = sum_j exp(s_j - m)
 *   out[i][t] = sum_j exp(s_j - m) * v[j][t] / l
 * Returns 0, or -1 if a scratch allocation fails.
 */
int oracle_attention_rows(const double *q, const double *k, const double *v,
                          int64_t S, int64_t d, double scale,
                          const int64_t *rows, int64_t n_rows, double *out)
{
    int failed = 0;
#pragma omp parallel
    {
        double *s = (double *)malloc((size_t)S * sizeof(double));
        if (!s) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < n_rows; ++r) {
            if (!s) continue;
            const int64_t i = rows[r];
            const double *qi = q + i * d;
            /* pass 1: scores and their maximum */
            double m = -INFINITY;
            for (int64_t j = 0; j < S; ++j) {
                const double *kj = k + j * d;
                double dot = 0.0;
                for (int64_t t = 0; t < d; ++t) dot += qi[t] * kj[t];
                s[j] = scale * dot;
                if (s[j] > m) m = s[j];
            }
            /* pass 2: exponentials, their sum, and the weighted sum of V rows */
            double *o = out + r * d;
            for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
            double l = 0.0;
            for (int64_t j = 0; j < S; ++j) {
                const double w = exp(s[j] - m);
                l += w;
                const double *vj = v + j * d;
                for (int64_t t = 0; t < d; ++t) o[t] += w * vj[t];
            }
            for (int64_t t = 0; t < d; ++t) o[t] /= l;
        }
        free(s);
    }
    return failed ? -1 : 0;
}

/*
 * Pack one head chunk.  src is [P][S/P][H][d] elements of elem_bytes bytes,
 * dst is [Hc][S][d].  Returns 0, or -1 on a shape the formula does not cover.
 */
int oracle_pack(const void *src, void *dst, int64_t P, int64_t S, int64_t H,
                int64_t d, int64_t h0, int64_t Hc, int64_t elem_bytes)
{
    if (P <= 0 || S % P != 0 || h0 < 0 || Hc < 0 || h0 + Hc > H) return -1;
    const int64_t Ss = S / P;
    const unsigned char *sp = (const unsigned char *)src;
    unsigned char *dp = (unsigned char *)dst;
    for (int64_t p = 0; p < P; ++p)
        for (int64_t s = 0; s < Ss; ++s)
            for (int64_t j = 0; j < Hc; ++j)
                for (int64_t e = 0; e < d; ++e) {
                    const int64_t from = ((p * Ss + s) * H + (h0 + j)) * d + e;
                    const int64_t to = (j * S + (p * Ss + s)) * d + e;
                    memcpy(dp + to * elem_bytes, sp + from * elem_bytes, (size_t)elem_bytes);
                }
    return 0;
}

/*
 * Unpack one head chunk.  src is [Hc][S][d], dst is [P][S/P][H][d]; only the
 * head slots [h0, h0+Hc) of dst are written.
 */
int oracle_unpack(const void *src, void *dst, int64_t P, int64_t S, int64_t H,
                  int64_t d, int64_t h0, int64_t Hc, int64_t elem_bytes)
{
    if (P <= 0 || S % P != 0 || h0 < 0 || Hc < 0 || h0 + Hc > H) return -1;
    const int64_t Ss = S / P;
    const unsigned char *sp = (const unsigned char *)src;
    unsigned char *dp = (unsigned char *)dst;
    for (int64_t p = 0; p < P; ++p)
        for (int64_t s = 0; s < Ss; ++s)
            for (int64_t j = 0; j < Hc; ++j)
                for (int64_t e = 0; e < d; ++e) {
                    const int64_t from = (j * S + (p * Ss + s)) * d + e;
                    const int64_t to = ((p * Ss + s) * H + (h0 + j)) * d + e;
                    memcpy(dp + to * elem_bytes, sp + from * elem_bytes, (size_t)elem_bytes);
                }
    return 0;
}

/*
 * Backward of one head.  With g = dL/dO (the output gradient):
 *   s_ij  = scale * <q_i, k_j>
 *   p_ij  = exp(s_ij - m_i) / l_i,  m_i = max_j s_ij,  l_i = sum_j exp(s_ij - m_i)
 *   dv_j  = sum_i p_ij g_i                      (O = P V)
 *   dp_ij = <g_i, v_j>
 *   ds_ij = p_ij (dp_ij - sum_k p_ik dp_ik)     (Jacobian of the row softmax)
 *   dq_i  = scale * sum_j ds_ij k_j
 *   dk_j  = scale * sum_i ds_ij q_i
 *   q, k, v, g : [S][d] row-major fp64
 *   q_rows     : n_q query indices whose dq is written to dq [n_q][d]
 *   k_rows     : n_k key indices whose dk, dv are written to dk, dv [n_k][d]
 * Pass 1 visits every query that a requested output needs (all of them when
 * n_k > 0) and keeps m_i, l_i and c_i = sum_k p_ik dp_ik; pass 2 sums over
 * all queries for each requested key.  Returns 0, or -1 if an allocation
 * fails.
 */
int oracle_attention_backward(const double *q, const double *k, const double *v, const double *g,
                              int64_t S, int64_t d, double scale,
                              const int64_t *q_rows, int64_t n_q,
                              const int64_t *k_rows, int64_t n_k,
                              double *dq, double *dk, double *dv)
{
    double *m = (double *)malloc((size_t)S * sizeof(double));
    double *l = (double *)malloc((size_t)S * sizeof(double));
    double *cdp = (double *)malloc((size_t)S * sizeof(double));
    int64_t *qpos = (int64_t *)malloc((size_t)S * sizeof(int64_t));
    if (!m || !l || !cdp || !qpos) {
        free(m); free(l); free(cdp); free(qpos);
        return -1;
    }
    /* qpos[i]: where query i's dq goes, or -1 */
    for (int64_t i = 0; i < S; ++i) qpos[i] = -1;
    for (int64_t r = 0; r < n_q; ++r) qpos[q_rows[r]] = r;
    int failed = 0;

    /* pass 1: per query row */
#pragma omp parallel
    {
        double *s = (double *)malloc((size_t)S * sizeof(double));
        double *dp = (double *)malloc((size_t)S * sizeof(double));
        if (!s || !dp) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < S; ++i) {
            if (!s || !dp) continue;
            if (n_k == 0 && qpos[i] < 0) continue;
            const double *qi = q + i * d, *gi = g + i * d;
            double mi = -INFINITY;
            for (int64_t j = 0; j < S; ++j) {
                double dot = 0.0, dg = 0.0;
                for (int64_t t = 0; t < d; ++t) {
                    dot += qi[t] * k[j * d + t];
                    dg += gi[t] * v[j * d + t];
                }
                s[j] = scale * dot;
                dp[j] = dg;
                if (s[j] > mi) mi = s[j];
            }
            double li = 0.0;
            for (int64_t j = 0; j < S; ++j) li += exp(s[j] - mi);
            double ci = 0.0;
            for (int64_t j = 0; j < S; ++j) ci += exp(s[j] - mi) / li * dp[j];
            m[i] = mi;
            l[i] = li;
            cdp[i] = ci;
            if (qpos[i] >= 0) {
                double *o = dq + qpos[i] * d;
                for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
                for (int64_t j = 0; j < S; ++j) {
                    const double ds = exp(s[j] - mi) / li * (dp[j] - ci);
                    for (int64_t t = 0; t < d; ++t) o[t] += scale * ds * k[j * d + t];
                }
            }
        }
        free(s);
        free(dp);
    }

    /* pass 2: per requested key row, summing over every query */
    if (!failed) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t r = 0; r < n_k; ++r) {
            const int64_t j = k_rows[r];
            const double *kj = k + j * d, *vj = v + j * d;
            double *okk = dk + r * d, *ov = dv + r * d;
            for (int64_t t = 0; t < d; ++t) okk[t] = ov[t] = 0.0;
            for (int64_t i = 0; i < S; ++i) {
                const double *qi = q + i * d, *gi = g + i * d;
                double dot = 0.0, dg = 0.0;
                for (int64_t t = 0; t < d; ++t) {
                    dot += qi[t] * kj[t];
                    dg += gi[t] * vj[t];
                }
                const double p = exp(scale * dot - m[i]) / l[i];
                const double ds = p * (dg - cdp[i]);
                for (int64_t t = 0; t < d; ++t) {
                    ov[t] += p * gi[t];
                    okk[t] += scale * ds * qi[t];
                }
            }
        }
    }
    free(m); free(l); free(cdp); free(qpos);
    return failed ? -1 : 0;
}

/* Number of OpenMP threads the attention oracle runs on (for reporting). */
int oracle_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
