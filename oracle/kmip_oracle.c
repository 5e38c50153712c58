/*
 * k-MIP self-attention: CPU oracle in float64.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow definition of what
 * the GPU path computes.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load it; the product library never
 * links, calls or falls back to it, and the two share no source.
 *
 * What is computed (arXiv 2604.03815):
 *   - Eq. (1), Section 3.1: per head h, A^h = softmax(scale * T_k(Q K^T)),
 *     where T_k keeps the k largest entries of each row and sets the rest
 *     to -inf.  The caller passes `scale` (the paper uses 1/sqrt(d_K)).
 *   - Algorithm 1 (Appendix E): SymbolicMultiply forms S = Q K^T,
 *     RowwiseTopK returns the k best indices and their scores per row,
 *     GatherRows picks the value rows, softmax runs over the k kept scores,
 *     and an einsum sums the weighted value rows.
 *   - Appendix F: the symbolic matrix entry is E_ij = q_i . k_j.
 *   - Attention dropout (the experimental details list an attention-dropout
 *     rate r): each kept weight A_ij is multiplied by m_ij / (1 - r) with a
 *     0/1 keep draw m_ij, inverted dropout as in Srivastava et al. (2014);
 *     the draws are an input (keep [.., k] uint8 aligned with the index
 *     slots, NULL for no dropout) so that both implementations see the same
 *     ones.  The softmax statistics (lse) are those of A, before dropout.
 *   - Backward (Section 3.1, last paragraph; Appendix E, last paragraph):
 *     the selected indices are reused, so gradients flow only through the
 *     k selected pairs of each query and the selection itself is constant.
 *     The paper prints no gradient formulas; they are the chain rule of
 *     Eq. (1) with the index set held fixed.
 *
 * Readings where the paper is silent:
 *   - ties: order by (score descending, key index ascending);
 *   - attention is restricted to the query's own graph [o_g, o_{g+1});
 *   - a graph with n < k nodes keeps all n keys, unused slots hold -1;
 *   - the query's own key is a candidate (no diagonal mask);
 *   - scale must be > 0, so selecting on raw scores equals selecting on
 *     scaled scores.
 *
 * All inputs are float64 arrays, node-major (row i, head h, dim t at
 * ((i * H) + h) * width + t): Q and K [N, H, d] with d = d_K, V and dO
 * [N, H, dv] with dv = d_V (Section 3.1 lets the value width differ from the
 * query/key width: W_V maps to d_V dimensions, W_Q and W_K to d_K).  Exact
 * bf16 values widen to float64 without rounding, so the oracle sees the same
 * numbers as the GPU path.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    double s;
    int32_t j;
} oracle_pair;

/* Total order of RowwiseTopK: larger score first, lower key index on ties. */
static int oracle_pair_order(const void* a, const void* b) {
    const oracle_pair* x = (const oracle_pair*)a;
    const oracle_pair* y = (const oracle_pair*)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->j > y->j) - (x->j < y->j);
}

static int oracle_int_order(const void* a, const void* b) {
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

/* Graph [lo, hi) that node i belongs to.  offsets == NULL means one graph. */
static void oracle_graph_range(const int32_t* offsets, int32_t G, int64_t N, int64_t i,
                               int64_t* lo, int64_t* hi) {
    if (offsets == NULL) {
        *lo = 0;
        *hi = N;
        return;
    }
    int32_t a = 0, b = G; /* find g with offsets[g] <= i < offsets[g+1] */
    while (b - a > 1) {
        int32_t m = (a + b) / 2;
        if (offsets[m] <= i) a = m; else b = m;
    }
    /* skip empty graphs that share the same start */
    while (a + 1 < G && offsets[a + 1] <= i) a++;
    *lo = offsets[a];
    *hi = offsets[a + 1];
}

/* Appendix F: E_ij = q_i . k_j for head h, summed over t = 0..d-1 in order. */
static double oracle_score(const double* Q, const double* K, int32_t H, int32_t d,
                           int64_t i, int64_t j, int32_t h) {
    const double* q = Q + ((size_t)i * H + h) * d;
    const double* kr = K + ((size_t)j * H + h) * d;
    double s = 0.0;
    for (int32_t t = 0; t < d; ++t) s += q[t] * kr[t];
    return s;
}

/*
 * RowwiseTopK (Algorithm 1) for selected query-heads.  Each row is sorted in
 * full by (score desc, index asc) and the first min(k, n) entries are kept.
 *   sel      query-head ids (i * H + h); NULL selects all N*H in order
 *   idx_out  [nsel, k] int32, unused slots -1
 *   s_out    [nsel, k] scores of the kept entries, unused slots -inf
 *   next_out [nsel] score of the (k+1)-th entry, -inf if n <= k
 * Returns 0, or -1 if a work buffer could not be allocated.
 */
int oracle_topk(const double* Q, const double* K, const int32_t* offsets, int32_t G,
                int64_t N, int32_t H, int32_t d, int32_t k, int64_t nsel, const int64_t* sel,
                int32_t* idx_out, double* s_out, double* next_out) {
    if (sel == NULL) nsel = N * (int64_t)H;
    int failed = 0;
#pragma omp parallel
    {
        oracle_pair* row = NULL;
        int64_t cap = 0;
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t qh = sel ? sel[r] : r;
            int64_t i = qh / H;
            int32_t h = (int32_t)(qh % H);
            int64_t lo, hi;
            oracle_graph_range(offsets, G, N, i, &lo, &hi);
            int64_t n = hi - lo;
            if (n > cap) {
                free(row);
                row = (oracle_pair*)malloc(sizeof(oracle_pair) * (size_t)n);
                cap = row ? n : 0;
                if (!row) {
#pragma omp atomic write
                    failed = 1;
                    continue;
                }
            }
            for (int64_t j = lo; j < hi; ++j) {
                row[j - lo].s = oracle_score(Q, K, H, d, i, j, h);
                row[j - lo].j = (int32_t)j;
            }
            qsort(row, (size_t)n, sizeof(oracle_pair), oracle_pair_order);
            for (int32_t t = 0; t < k; ++t) {
                idx_out[r * k + t] = t < n ? row[t].j : -1;
                if (s_out) s_out[r * k + t] = t < n ? row[t].s : -INFINITY;
            }
            if (next_out) next_out[r] = n > k ? row[k].s : -INFINITY;
        }
        free(row);
    }
    return failed ? -1 : 0;
}

/*
 * Softmax over the kept scores and the weighted sum of gathered value rows
 * (Algorithm 1: GatherRows, softmax, Einsum nk,nkv->nv), for a given index
 * set.  Slots holding -1 are empty (their weight is exp(-inf) = 0).
 *   keep [nsel, k] (NULL: no dropout): the weight of slot t is multiplied
 *   by keep_scale when keep[t] != 0 and by 0 otherwise.
 *   out [nsel, dv], lse [nsel] (natural log of sum_j exp(scale * s_ij)).
 * A row with no valid index gets out = 0 and lse = -inf.
 */
int oracle_attend(const double* Q, const double* K, const double* V, int64_t N, int32_t H,
                  int32_t d, int32_t dv, int32_t k, double scale, int64_t nsel, const int64_t* sel,
                  const int32_t* idx, const uint8_t* keep, double keep_scale, double* out, double* lse) {
    if (sel == NULL) nsel = N * (int64_t)H;
#pragma omp parallel
    {
        double* z = (double*)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
#pragma omp for schedule(static)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t qh = sel ? sel[r] : r;
            int64_t i = qh / H;
            int32_t h = (int32_t)(qh % H);
            const int32_t* row = idx + r * k;
            double zmax = -INFINITY;
            for (int32_t t = 0; t < k; ++t) {
                z[t] = row[t] >= 0 ? scale * oracle_score(Q, K, H, d, i, row[t], h) : -INFINITY;
                if (z[t] > zmax) zmax = z[t];
            }
            double* o = out + r * dv;
            for (int32_t c = 0; c < dv; ++c) o[c] = 0.0;
            if (zmax == -INFINITY) {
                lse[r] = -INFINITY;
                continue;
            }
            double Z = 0.0;
            for (int32_t t = 0; t < k; ++t) Z += row[t] >= 0 ? exp(z[t] - zmax) : 0.0;
            for (int32_t t = 0; t < k; ++t) {
                if (row[t] < 0) continue;
                double p = exp(z[t] - zmax) / Z;
                if (keep) p *= keep[r * k + t] ? keep_scale : 0.0;
                const double* vr = V + ((size_t)row[t] * H + h) * dv;
                for (int32_t c = 0; c < dv; ++c) o[c] += p * vr[c];
            }
            lse[r] = zmax + log(Z);
        }
        free(z);
    }
    return 0;
}

/*
 * Full forward: RowwiseTopK for every query-head, then oracle_attend.
 * idx [N, H, k], out [N, H, dv], lse [N, H].
 */
int oracle_forward(const double* Q, const double* K, const double* V, const int32_t* offsets,
                   int32_t G, int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, double scale,
                   int32_t* idx, double* out, double* lse) {
    if (oracle_topk(Q, K, offsets, G, N, H, d, k, 0, NULL, idx, NULL, NULL) != 0) return -1;
    return oracle_attend(Q, K, V, N, H, d, dv, k, scale, 0, NULL, idx, NULL, 1.0, out, lse);
}

/*
 * Backward with the index set held fixed.  For each query i and head h,
 * with p_j the softmax weights over the kept keys j and dO_i the incoming
 * gradient of out_i:
 *   dp_j  = dO_i . v_j
 *   D_i   = sum_j p_j dp_j
 *   g_j   = p_j (dp_j - D_i)                 (gradient of the logit scale*s_ij)
 *   dQ_i  = sum_j g_j * scale * k_j
 *   dK_j += g_j * scale * q_i
 *   dV_j += p_j * dO_i
 * (the dot product dp_j runs over the dv value dimensions, dQ and dK have
 * the d query/key dimensions, dV the dv value dimensions).  With dropout
 * (keep [N, H, k] not NULL, f_j = keep_scale or 0 by keep), out_i sums
 * p_j f_j v_j, so dV_j gets p_j f_j dO_i and the gradient of p_j is
 * f_j dp_j, which replaces dp_j in D_i and g_j.
 * idx [N, H, k]; dQ, dK [N, H, d] and dV [N, H, dv] are overwritten.
 * Per-query terms are computed in parallel; the scatter into dK and dV runs
 * in one thread in query order.
 */
int oracle_backward(const double* Q, const double* K, const double* V, const double* dO,
                    int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, double scale,
                    const int32_t* idx, const uint8_t* keep, double keep_scale, double* dQ, double* dK,
                    double* dV) {
    int64_t NH = N * (int64_t)H;
    double* P = (double*)malloc(sizeof(double) * (size_t)(NH * k > 0 ? NH * k : 1));
    double* Gr = (double*)malloc(sizeof(double) * (size_t)(NH * k > 0 ? NH * k : 1));
    double* F = (double*)malloc(sizeof(double) * (size_t)(NH * k > 0 ? NH * k : 1));
    if (!P || !Gr || !F) {
        free(P);
        free(Gr);
        free(F);
        return -1;
    }
    memset(dQ, 0, sizeof(double) * (size_t)(NH * d));
    memset(dK, 0, sizeof(double) * (size_t)(NH * d));
    memset(dV, 0, sizeof(double) * (size_t)(NH * dv));
#pragma omp parallel
    {
        double* z = (double*)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
        double* dp = (double*)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
#pragma omp for schedule(static)
        for (int64_t qh = 0; qh < NH; ++qh) {
            int64_t i = qh / H;
            int32_t h = (int32_t)(qh % H);
            const int32_t* row = idx + qh * k;
            double* p = P + qh * k;
            double* g = Gr + qh * k;
            double* f = F + qh * k;
            for (int32_t t = 0; t < k; ++t) f[t] = keep ? (keep[qh * k + t] ? keep_scale : 0.0) : 1.0;
            double zmax = -INFINITY;
            for (int32_t t = 0; t < k; ++t) {
                z[t] = row[t] >= 0 ? scale * oracle_score(Q, K, H, d, i, row[t], h) : -INFINITY;
                if (z[t] > zmax) zmax = z[t];
            }
            if (zmax == -INFINITY) {
                for (int32_t t = 0; t < k; ++t) p[t] = g[t] = 0.0;
                continue;
            }
            double Z = 0.0;
            for (int32_t t = 0; t < k; ++t) Z += row[t] >= 0 ? exp(z[t] - zmax) : 0.0;
            const double* dOi = dO + (size_t)qh * dv;
            double D = 0.0;
            for (int32_t t = 0; t < k; ++t) {
                p[t] = row[t] >= 0 ? exp(z[t] - zmax) / Z : 0.0;
                dp[t] = 0.0;
                if (row[t] >= 0) {
                    const double* vr = V + ((size_t)row[t] * H + h) * dv;
                    for (int32_t c = 0; c < dv; ++c) dp[t] += dOi[c] * vr[c];
                    dp[t] *= f[t];
                }
                D += p[t] * dp[t];
            }
            double* dq = dQ + (size_t)qh * d;
            for (int32_t t = 0; t < k; ++t) {
                g[t] = p[t] * (dp[t] - D);
                if (row[t] < 0) continue;
                const double* kr = K + ((size_t)row[t] * H + h) * d;
                for (int32_t c = 0; c < d; ++c) dq[c] += g[t] * scale * kr[c];
            }
        }
        free(z);
        free(dp);
    }
    for (int64_t qh = 0; qh < NH; ++qh) {
        int32_t h = (int32_t)(qh % H);
        const int32_t* row = idx + qh * k;
        const double* qi = Q + (size_t)qh * d;
        const double* dOi = dO + (size_t)qh * dv;
        for (int32_t t = 0; t < k; ++t) {
            if (row[t] < 0) continue;
            double* dkr = dK + ((size_t)row[t] * H + h) * d;
            double* dvr = dV + ((size_t)row[t] * H + h) * dv;
            double gs = Gr[qh * k + t] * scale, pt = P[qh * k + t] * F[qh * k + t];
            for (int32_t c = 0; c < d; ++c) dkr[c] += gs * qi[c];
            for (int32_t c = 0; c < dv; ++c) dvr[c] += pt * dOi[c];
        }
    }
    free(P);
    free(Gr);
    free(F);
    return 0;
}

/*
 * Checks a candidate index set (e.g. one produced elsewhere) for the
 * selected query-heads against exact scores.
 *   min_in  [nsel] smallest exact score inside the set (+inf if empty)
 *   max_out [nsel] largest exact score of a graph key outside the set
 *                  (-inf if the set covers the graph)
 *   flags   [nsel] bit 1: index outside the query's graph
 *                  bit 2: duplicate index
 *                  bit 4: number of distinct valid entries != min(k, n)
 *                  bit 8: a -1 slot precedes a valid entry
 */
int oracle_check_set(const double* Q, const double* K, const int32_t* offsets, int32_t G,
                     int64_t N, int32_t H, int32_t d, int32_t k, int64_t nsel,
                     const int64_t* sel, const int32_t* idx, double* min_in, double* max_out,
                     int32_t* flags) {
    if (sel == NULL) nsel = N * (int64_t)H;
#pragma omp parallel
    {
        int32_t* set = (int32_t*)malloc(sizeof(int32_t) * (size_t)(k > 0 ? k : 1));
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t qh = sel ? sel[r] : r;
            int64_t i = qh / H;
            int32_t h = (int32_t)(qh % H);
            int64_t lo, hi;
            oracle_graph_range(offsets, G, N, i, &lo, &hi);
            int64_t n = hi - lo;
            const int32_t* row = idx + r * k;
            int32_t f = 0, m = 0, seen_pad = 0;
            double mn = INFINITY;
            for (int32_t t = 0; t < k; ++t) {
                if (row[t] < 0) {
                    seen_pad = 1;
                    continue;
                }
                if (seen_pad) f |= 8;
                if (row[t] < lo || row[t] >= hi) {
                    f |= 1;
                    continue;
                }
                set[m++] = row[t];
                double s = oracle_score(Q, K, H, d, i, row[t], h);
                if (s < mn) mn = s;
            }
            qsort(set, (size_t)m, sizeof(int32_t), oracle_int_order);
            int32_t distinct = m > 0 ? 1 : 0;
            for (int32_t t = 1; t < m; ++t) {
                if (set[t] == set[t - 1]) f |= 2;
                else distinct++;
            }
            int64_t want = n < k ? n : k;
            if (distinct != want) f |= 4;
            /* largest score of a graph key outside the set; membership is
               looked up only for a score that would raise the maximum */
            double mx = -INFINITY;
            for (int64_t j = lo; j < hi; ++j) {
                double s = oracle_score(Q, K, H, d, i, j, h);
                if (!(s > mx)) continue;
                int32_t jj = (int32_t)j;
                if (bsearch(&jj, set, (size_t)m, sizeof(int32_t), oracle_int_order)) continue;
                mx = s;
            }
            min_in[r] = mn;
            max_out[r] = mx;
            flags[r] = f;
        }
        free(set);
    }
    return 0;
}

/* Number of OpenMP threads the functions above use. */
int oracle_threads(void) { return omp_get_max_threads(); }
