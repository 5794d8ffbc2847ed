/*
 * evo_attn_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, fp64 reference implementation of the Evoformer gated
 * multi-head attention with pair bias, forward and analytic backward.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library; the product path never does.  It shares no code,
 * header or constant with the GPU library.
 *
 * What is computed (ScaleFold, Section 3.3 "Multi Head Attention": AlphaFold's
 * attention variant adds a pair-bias term to the logits before the softmax,
 * and the fused kernel is FlashAttention-based, i.e. an exact rewrite of the
 * plain softmax attention written out below).  For row r (bias plane
 * b = r / rows_per_bias), head h, query i, key j, channel c:
 *
 *   s[i][j]  = (1/sqrt(d)) * sum_c q[r,i,h,c] * k[r,j,h,c] + bias[b,h,i,j]
 *   P[i][j]  = softmax over the kept keys j (key_mask[r,j] != 0) of s[i][.],
 *              0 for masked keys
 *   a[i][c]  = sum_j P[i][j] * v[r,j,h,c]
 *   o        = sigmoid(g) * a           (sigmoid == 1 when there is no gate)
 *   lse[i]   = log(sum_{kept j} exp(s[i][j]))   (natural log)
 *
 * A query whose keys are all masked has o = 0, lse = -inf and zero gradients.
 *
 * Backward (chain rule through the definitions above; dO = dL/do):
 *   dA      = dO * sigmoid(g)
 *   dG      = dO * a * sigmoid(g) * (1 - sigmoid(g))
 *   dV[j]  += sum_i P[i][j] * dA[i]
 *   dP[i][j] = dA[i] . v[j]
 *   dS[i][j] = P[i][j] * (dP[i][j] - sum_k P[i][k] * dP[i][k])  (softmax Jacobian)
 *   dQ[i]   = (1/sqrt(d)) * sum_j dS[i][j] * k[j]
 *   dK[j]   = (1/sqrt(d)) * sum_i dS[i][j] * q[i]
 *   dBias[b,h,i,j] = sum over the rows r of plane b of dS[i][j]
 *
 * Layouts (all contiguous, fp64): q,k,v,g,o,dO,dq,dk,dv,dg are [N][L][H][d];
 * bias and dbias are [B][H][L][L] with B = N / rows_per_bias; key_mask is
 * [N][L] bytes (nonzero = keep); lse is [N][H][L].
 *
 * Parallelism: OpenMP over (row, head) pairs, each owning a private L x L
 * scratch; the backward keeps one dBias accumulator per thread and adds them
 * up at the end.  No blocking, fusion or reordering beyond that.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int64_t n_rows;        /* N */
    int64_t seq_len;       /* L */
    int64_t n_heads;       /* H */
    int64_t head_dim;      /* d */
    int64_t rows_per_bias; /* rows sharing one bias plane */
} evo_oracle_dims;

enum { ORACLE_OK = 0, ORACLE_BAD_ARG = 1, ORACLE_NO_MEMORY = 2 };

static int check_dims(const evo_oracle_dims *dm) {
    if (!dm) return ORACLE_BAD_ARG;
    if (dm->n_rows < 0 || dm->seq_len < 0 || dm->n_heads <= 0 || dm->head_dim <= 0)
        return ORACLE_BAD_ARG;
    if (dm->rows_per_bias <= 0 || dm->n_rows % dm->rows_per_bias != 0) return ORACLE_BAD_ARG;
    return ORACLE_OK;
}

/* index of element (r, t, h, c) in a [N][L][H][d] tensor */
static inline int64_t tok_index(const evo_oracle_dims *dm, int64_t r, int64_t t, int64_t h,
                                int64_t c) {
    return ((r * dm->seq_len + t) * dm->n_heads + h) * dm->head_dim + c;
}

static inline double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/*
 * Softmax probabilities of one (row, head): P[i*L + j].
 * Returns, through lse (length L, may be NULL), the log-sum-exp of each query.
 */
static void probs_one(const evo_oracle_dims *dm, const double *q, const double *k,
                      const double *bias, const uint8_t *mask, int64_t r, int64_t h,
                      double *P, double *lse) {
    const int64_t L = dm->seq_len, d = dm->head_dim;
    const double scale = 1.0 / sqrt((double)d);
    const int64_t b = r / dm->rows_per_bias;
    for (int64_t i = 0; i < L; ++i) {
        double *row = P + i * L;
        double m = -INFINITY;
        for (int64_t j = 0; j < L; ++j) {
            int keep = mask ? (mask[r * L + j] != 0) : 1;
            if (!keep) {
                row[j] = -INFINITY;
                continue;
            }
            double dot = 0.0;
            for (int64_t c = 0; c < d; ++c)
                dot += q[tok_index(dm, r, i, h, c)] * k[tok_index(dm, r, j, h, c)];
            double s = scale * dot;
            if (bias) s += bias[((b * dm->n_heads + h) * L + i) * L + j];
            row[j] = s;
            if (s > m) m = s;
        }
        if (m == -INFINITY) {
            /* every key masked: the row contributes nothing */
            for (int64_t j = 0; j < L; ++j) row[j] = 0.0;
            if (lse) lse[i] = -INFINITY;
            continue;
        }
        double sum = 0.0;
        for (int64_t j = 0; j < L; ++j) {
            double e = (row[j] == -INFINITY) ? 0.0 : exp(row[j] - m);
            row[j] = e;
            sum += e;
        }
        for (int64_t j = 0; j < L; ++j) row[j] /= sum;
        if (lse) lse[i] = m + log(sum);
    }
}

int evo_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* P of one (row, head), for invariant checks.  P has L*L entries. */
int evo_oracle_probs(const evo_oracle_dims *dm, const double *q, const double *k,
                     const double *bias, const uint8_t *mask, int64_t r, int64_t h, double *P) {
    int st = check_dims(dm);
    if (st) return st;
    if (!q || !k || !P || r < 0 || r >= dm->n_rows || h < 0 || h >= dm->n_heads)
        return ORACLE_BAD_ARG;
    probs_one(dm, q, k, bias, mask, r, h, P, NULL);
    return ORACLE_OK;
}

int evo_oracle_fwd(const evo_oracle_dims *dm, const double *q, const double *k, const double *v,
                   const double *g, const double *bias, const uint8_t *mask, double *out,
                   double *lse) {
    int st = check_dims(dm);
    if (st) return st;
    if (!q || !k || !v || !out || !lse) return ORACLE_BAD_ARG;
    const int64_t N = dm->n_rows, L = dm->seq_len, H = dm->n_heads, d = dm->head_dim;
    if (N == 0 || L == 0) return ORACLE_OK;
    int failed = 0;
#pragma omp parallel
    {
        double *P = (double *)malloc(sizeof(double) * (size_t)(L * L));
        if (!P) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic)
        for (int64_t rh = 0; rh < N * H; ++rh) {
            if (!P) continue;
            const int64_t r = rh / H, h = rh % H;
            probs_one(dm, q, k, bias, mask, r, h, P, lse + (r * H + h) * L);
            for (int64_t i = 0; i < L; ++i) {
                for (int64_t c = 0; c < d; ++c) {
                    double a = 0.0;
                    for (int64_t j = 0; j < L; ++j) a += P[i * L + j] * v[tok_index(dm, r, j, h, c)];
                    const int64_t x = tok_index(dm, r, i, h, c);
                    out[x] = g ? sigmoid(g[x]) * a : a;
                }
            }
        }
        free(P);
    }
    return failed ? ORACLE_NO_MEMORY : ORACLE_OK;
}

int evo_oracle_bwd(const evo_oracle_dims *dm, const double *q, const double *k, const double *v,
                   const double *g, const double *bias, const uint8_t *mask, const double *dout,
                   double *dq, double *dk, double *dv, double *dg, double *dbias) {
    int st = check_dims(dm);
    if (st) return st;
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return ORACLE_BAD_ARG;
    if ((g == NULL) != (dg == NULL) || (bias == NULL) != (dbias == NULL)) return ORACLE_BAD_ARG;
    const int64_t N = dm->n_rows, L = dm->seq_len, H = dm->n_heads, d = dm->head_dim;
    const int64_t B = N / dm->rows_per_bias;
    const double scale = 1.0 / sqrt((double)d);
    const size_t tok_elems = (size_t)(N * L * H * d);
    const size_t bias_elems = (size_t)(B * H * L * L);
    memset(dq, 0, sizeof(double) * tok_elems);
    memset(dk, 0, sizeof(double) * tok_elems);
    memset(dv, 0, sizeof(double) * tok_elems);
    if (dg) memset(dg, 0, sizeof(double) * tok_elems);
    if (dbias) memset(dbias, 0, sizeof(double) * bias_elems);
    if (N == 0 || L == 0) return ORACLE_OK;
    int failed = 0;
#pragma omp parallel
    {
        double *P = (double *)malloc(sizeof(double) * (size_t)(L * L));
        double *dS = (double *)malloc(sizeof(double) * (size_t)(L * L));
        double *dA = (double *)malloc(sizeof(double) * (size_t)(L * d));
        double *my_dbias = dbias ? (double *)calloc(bias_elems, sizeof(double)) : NULL;
        int ok = P && dS && dA && (!dbias || my_dbias);
        if (!ok) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic)
        for (int64_t rh = 0; rh < N * H; ++rh) {
            if (!ok) continue;
            const int64_t r = rh / H, h = rh % H, b = r / dm->rows_per_bias;
            probs_one(dm, q, k, bias, mask, r, h, P, NULL);
            /* attention output before the gate, and the gate's two gradients */
            for (int64_t i = 0; i < L; ++i) {
                for (int64_t c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (int64_t j = 0; j < L; ++j) acc += P[i * L + j] * v[tok_index(dm, r, j, h, c)];
                    const int64_t x = tok_index(dm, r, i, h, c);
                    if (g) {
                        const double sg = sigmoid(g[x]);
                        dA[i * d + c] = dout[x] * sg;
                        dg[x] = dout[x] * acc * sg * (1.0 - sg);
                    } else {
                        dA[i * d + c] = dout[x];
                    }
                }
            }
            /* dV[j] = sum_i P[i][j] dA[i] */
            for (int64_t j = 0; j < L; ++j)
                for (int64_t c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (int64_t i = 0; i < L; ++i) acc += P[i * L + j] * dA[i * d + c];
                    dv[tok_index(dm, r, j, h, c)] = acc;
                }
            /* dP, then the softmax Jacobian applied row by row */
            for (int64_t i = 0; i < L; ++i) {
                double *dPi = dS + i * L;
                for (int64_t j = 0; j < L; ++j) {
                    double acc = 0.0;
                    for (int64_t c = 0; c < d; ++c) acc += dA[i * d + c] * v[tok_index(dm, r, j, h, c)];
                    dPi[j] = acc;
                }
                double pdp = 0.0;
                for (int64_t j = 0; j < L; ++j) pdp += P[i * L + j] * dPi[j];
                for (int64_t j = 0; j < L; ++j) dPi[j] = P[i * L + j] * (dPi[j] - pdp);
            }
            /* dQ, dK */
            for (int64_t i = 0; i < L; ++i)
                for (int64_t c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (int64_t j = 0; j < L; ++j) acc += dS[i * L + j] * k[tok_index(dm, r, j, h, c)];
                    dq[tok_index(dm, r, i, h, c)] = scale * acc;
                }
            for (int64_t j = 0; j < L; ++j)
                for (int64_t c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (int64_t i = 0; i < L; ++i) acc += dS[i * L + j] * q[tok_index(dm, r, i, h, c)];
                    dk[tok_index(dm, r, j, h, c)] = scale * acc;
                }
            /* this row's contribution to the shared bias plane */
            if (my_dbias) {
                double *plane = my_dbias + (b * H + h) * L * L;
                for (int64_t x = 0; x < L * L; ++x) plane[x] += dS[x];
            }
        }
        if (my_dbias && ok) {
#pragma omp critical
            for (size_t x = 0; x < bias_elems; ++x) dbias[x] += my_dbias[x];
        }
        free(P);
        free(dS);
        free(dA);
        free(my_dbias);
    }
    return failed ? ORACLE_NO_MEMORY : ORACLE_OK;
}
