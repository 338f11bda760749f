/*
 * Exact attention forward and vector-Jacobian product in FP64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the tests, the smoke check and the CPU baseline leg
 * of the benchmark use it.
 *
 * What it computes (paper, Section 3.2, eqs. row-attention and row-gradients):
 * for each query row i with support L_i (j <= i when causal, all j otherwise)
 *     s_ij = alpha q_i.k_j,   p_ij = softmax_j(s_ij),   o_i = sum_j p_ij v_j
 *     a_ij = u_i.v_j,  mu_a = sum_j p_ij a_ij,  g_ij = p_ij (a_ij - mu_a)
 *     dq_i = alpha sum_j g_ij k_j,  dk_j = alpha sum_i g_ij q_i,  dv_j = sum_i p_ij u_i
 * with u = dO.  The paper measures errors against this VJP in FP64 on the same
 * BF16 inputs (Section 3.2; appendix "Reference and metric": centered scores
 * and values).  Following that appendix, scores and values are centered first:
 * the per-head key mean kbar and value mean vbar are subtracted.  Softmax is
 * unchanged by the row constant alpha q_i.kbar, and g is unchanged by a common
 * value shift (Proposition 3.1, exact translation structure), so this is the
 * same mathematical quantity computed with less cancellation:
 *     st_ij = alpha q_i.(k_j - kbar)
 *     LSE_i = alpha q_i.kbar + max_j st_ij + ln sum_j exp(st_ij - max)
 *     ot_i  = sum_j p_ij (v_j - vbar),   o_i = vbar + ot_i
 *     c_ij  = u_i.((v_j - vbar) - ot_i)          (= a_ij - mu_a, exactly)
 *     dq_i  = alpha sum_j p_ij (kt_j - mut_i) c_ij, mut_i = sum_j p_ij kt_j
 *             (the covariance form of Proposition 3.1)
 * LSE is in natural-log units of the scaled scores.
 *
 * Two phases per head: rows in parallel (O, LSE, dQ and the row statistics),
 * then key columns in parallel (dK, dV), recomputing p_ij and c_ij with the
 * same expressions.  No tiling, fusion or reordering beyond that.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double dot(const double* a, const double* b, int64_t d) {
    double s = 0.0;
    for (int64_t c = 0; c < d; ++c) s += a[c] * b[c];
    return s;
}

/* u.((vt_j) - ot) without forming the difference vector separately. */
static double dot_diff(const double* u, const double* vt, const double* ot, int64_t d) {
    double s = 0.0;
    for (int64_t c = 0; c < d; ++c) s += u[c] * (vt[c] - ot[c]);
    return s;
}

static int one_head(int64_t N, int64_t d, int causal, double alpha,
                    const double* q, const double* k, const double* v, const double* u,
                    double* o, double* lse, double* dq, double* dk, double* dv) {
    double* kbar = calloc((size_t)d, sizeof(double));
    double* vbar = calloc((size_t)d, sizeof(double));
    double* kt = malloc((size_t)(N * d) * sizeof(double));
    double* vt = malloc((size_t)(N * d) * sizeof(double));
    double* ot = malloc((size_t)(N * d) * sizeof(double));
    double* rowM = malloc((size_t)N * sizeof(double));
    double* rowZ = malloc((size_t)N * sizeof(double));
    if (!kbar || !vbar || !kt || !vt || !ot || !rowM || !rowZ) {
        free(kbar); free(vbar); free(kt); free(vt); free(ot); free(rowM); free(rowZ);
        return 1;
    }
    for (int64_t j = 0; j < N; ++j)
        for (int64_t c = 0; c < d; ++c) {
            kbar[c] += k[j * d + c];
            vbar[c] += v[j * d + c];
        }
    for (int64_t c = 0; c < d; ++c) {
        kbar[c] /= (double)N;
        vbar[c] /= (double)N;
    }
    for (int64_t j = 0; j < N; ++j)
        for (int64_t c = 0; c < d; ++c) {
            kt[j * d + c] = k[j * d + c] - kbar[c];
            vt[j * d + c] = v[j * d + c] - vbar[c];
        }

    int fail = 0;
    /* Phase 1: one query row at a time. */
#pragma omp parallel reduction(| : fail)
    {
        double* s = malloc((size_t)N * sizeof(double));
        double* p = malloc((size_t)N * sizeof(double));
        double* cc = malloc((size_t)N * sizeof(double));
        double* mu = malloc((size_t)d * sizeof(double));
        if (!s || !p || !cc || !mu) {
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 8)
            for (int64_t i = 0; i < N; ++i) {
                const double* qi = q + i * d;
                const double* ui = u + i * d;
                int64_t L = causal ? i + 1 : N;
                double M = -INFINITY;
                for (int64_t j = 0; j < L; ++j) {
                    s[j] = alpha * dot(qi, kt + j * d, d);
                    if (s[j] > M) M = s[j];
                }
                double Z = 0.0;
                for (int64_t j = 0; j < L; ++j) Z += exp(s[j] - M);
                for (int64_t j = 0; j < L; ++j) p[j] = exp(s[j] - M) / Z;
                double* oti = ot + i * d;
                for (int64_t c = 0; c < d; ++c) { oti[c] = 0.0; mu[c] = 0.0; }
                for (int64_t j = 0; j < L; ++j)
                    for (int64_t c = 0; c < d; ++c) {
                        oti[c] += p[j] * vt[j * d + c];
                        mu[c] += p[j] * kt[j * d + c];
                    }
                for (int64_t c = 0; c < d; ++c) o[i * d + c] = vbar[c] + oti[c];
                lse[i] = alpha * dot(qi, kbar, d) + M + log(Z);
                rowM[i] = M;
                rowZ[i] = Z;
                for (int64_t j = 0; j < L; ++j) cc[j] = dot_diff(ui, vt + j * d, oti, d);
                double* dqi = dq + i * d;
                for (int64_t c = 0; c < d; ++c) dqi[c] = 0.0;
                for (int64_t j = 0; j < L; ++j) {
                    double w = p[j] * cc[j];
                    for (int64_t c = 0; c < d; ++c) dqi[c] += w * (kt[j * d + c] - mu[c]);
                }
                for (int64_t c = 0; c < d; ++c) dqi[c] *= alpha;
            }
        }
        free(s); free(p); free(cc); free(mu);
    }

    /* Phase 2: one key column at a time. */
    if (!fail) {
#pragma omp parallel for schedule(dynamic, 8)
        for (int64_t j = 0; j < N; ++j) {
            double* dkj = dk + j * d;
            double* dvj = dv + j * d;
            for (int64_t c = 0; c < d; ++c) { dkj[c] = 0.0; dvj[c] = 0.0; }
            for (int64_t i = causal ? j : 0; i < N; ++i) {
                const double* qi = q + i * d;
                const double* ui = u + i * d;
                double sij = alpha * dot(qi, kt + j * d, d);
                double pij = exp(sij - rowM[i]) / rowZ[i];
                double gij = pij * dot_diff(ui, vt + j * d, ot + i * d, d);
                for (int64_t c = 0; c < d; ++c) {
                    dkj[c] += gij * qi[c];
                    dvj[c] += pij * ui[c];
                }
            }
            for (int64_t c = 0; c < d; ++c) dkj[c] *= alpha;
        }
    }
    free(kbar); free(vbar); free(kt); free(vt); free(ot); free(rowM); free(rowZ);
    return fail;
}

/*
 * BH heads laid out as [BH][N][d] (row-major, d innermost), LSE as [BH][N].
 * Returns 0 on success, 1 on allocation failure, 2 on bad arguments.
 */
/* nthreads > 0 runs the call on that many OpenMP threads and restores the
 * previous setting afterwards; 0 keeps the current setting. */
static int push_threads(int nthreads) {
#ifdef _OPENMP
    const int prev = omp_get_max_threads();
    if (nthreads > 0) omp_set_num_threads(nthreads);
    return prev;
#else
    (void)nthreads;
    return 1;
#endif
}

static void pop_threads(int prev) {
#ifdef _OPENMP
    omp_set_num_threads(prev);
#else
    (void)prev;
#endif
}

static int attention_heads(int64_t BH, int64_t N, int64_t d, int causal, double alpha,
                           const double* Q, const double* K, const double* V, const double* dO,
                           double* O, double* LSE, double* dQ, double* dK, double* dV) {
    for (int64_t h = 0; h < BH; ++h) {
        int64_t off = h * N * d;
        if (N == 0) continue;
        if (one_head(N, d, causal, alpha, Q + off, K + off, V + off, dO + off,
                     O + off, LSE + h * N, dQ + off, dK + off, dV + off))
            return 1;
    }
    return 0;
}

int oracle_attention_f64(int64_t BH, int64_t N, int64_t d, int causal, double alpha,
                         const double* Q, const double* K, const double* V, const double* dO,
                         double* O, double* LSE, double* dQ, double* dK, double* dV,
                         int nthreads) {
    if (BH < 0 || N < 0 || d < 1) return 2;
    const int prev = push_threads(nthreads);
    const int rc = attention_heads(BH, N, d, causal, alpha, Q, K, V, dO, O, LSE, dQ, dK, dV);
    pop_threads(prev);
    return rc;
}

/*
 * Grouped-query attention: Q, dO, O, dQ are [B][Hq][N][d], K, V, dK, dV are
 * [B][Hkv][N][d], LSE is [B][Hq][N], and query head h of batch b reads key/value
 * head h / (Hq / Hkv).  Each query head's VJP is the multi-head one above; the
 * key and value gradients of a key/value head are the sums of its query heads'
 * contributions (paper, Section 3.2 after eq. row-gradients: key and value
 * contributions also sum over the query heads that share a KV head), added in
 * head order.  Returns 0, 1 (allocation failure) or 2 (bad arguments).
 */
static int attention_gqa(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d, int causal,
                         double alpha, const double* Q, const double* K, const double* V,
                         const double* dO, double* O, double* LSE, double* dQ, double* dK,
                         double* dV) {
    const int64_t G = Hq / Hkv, hd = N * d;
    memset(dK, 0, (size_t)(B * Hkv * hd) * sizeof(double));
    memset(dV, 0, (size_t)(B * Hkv * hd) * sizeof(double));
    if (N == 0) return 0;
    double* tk = malloc((size_t)hd * sizeof(double));
    double* tv = malloc((size_t)hd * sizeof(double));
    if (!tk || !tv) {
        free(tk); free(tv);
        return 1;
    }
    for (int64_t b = 0; b < B; ++b)
        for (int64_t h = 0; h < Hq; ++h) {
            const int64_t qh = b * Hq + h, kh = b * Hkv + h / G;
            if (one_head(N, d, causal, alpha, Q + qh * hd, K + kh * hd, V + kh * hd, dO + qh * hd,
                         O + qh * hd, LSE + qh * N, dQ + qh * hd, tk, tv)) {
                free(tk); free(tv);
                return 1;
            }
            for (int64_t e = 0; e < hd; ++e) {
                dK[kh * hd + e] += tk[e];
                dV[kh * hd + e] += tv[e];
            }
        }
    free(tk); free(tv);
    return 0;
}

int oracle_attention_gqa_f64(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d, int causal,
                             double alpha, const double* Q, const double* K, const double* V,
                             const double* dO, double* O, double* LSE, double* dQ, double* dK,
                             double* dV, int nthreads) {
    if (B < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || N < 0 || d < 1) return 2;
    const int prev = push_threads(nthreads);
    const int rc = attention_gqa(B, Hq, Hkv, N, d, causal, alpha, Q, K, V, dO, O, LSE, dQ, dK, dV);
    pop_threads(prev);
    return rc;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
