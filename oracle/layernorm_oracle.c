/*
 * layernorm_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain fp64 reference of the LayerNorm that precedes every Evoformer
 * attention and transition block, forward and analytic backward.  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load
 * this library; the product path never does, and this file shares no code,
 * header or constant with the GPU library.
 *
 * What is computed (ScaleFold, Section 3.3, "LayerNormalization": the
 * paper's kernel changes how the work is spread over the GPU and how the
 * statistics and the parameter-gradient sums are gathered, not the
 * operation, which is the usual layer normalisation over the last axis).
 * For row r of an [R][C] input and channel c:
 *
 *   mean[r] = (1/C) sum_c x[r][c]
 *   var[r]  = (1/C) sum_c (x[r][c] - mean[r])^2        (biased variance)
 *   rstd[r] = 1 / sqrt(var[r] + eps)
 *   y[r][c] = (x[r][c] - mean[r]) * rstd[r] * w[c] + b[c]
 *
 * Backward (chain rule through the lines above; dy = dL/dy), with
 * xhat = (x - mean) * rstd and gx = dy * w:
 *
 *   dx[r][c] = rstd[r] * (gx[r][c] - (1/C) sum_k gx[r][k]
 *                         - xhat[r][c] * (1/C) sum_k gx[r][k] xhat[r][k])
 *   dw[c]    = sum_r dy[r][c] * xhat[r][c]
 *   db[c]    = sum_r dy[r][c]
 *
 * The backward recomputes mean and rstd from x (it does not trust saved
 * statistics).  The two means and the variance are each a separate loop over
 * the row, in channel order; the parameter sums run over rows in order.
 * OpenMP splits rows for x and y; the dw/db sums stay sequential.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

enum { LN_OK = 0, LN_BAD_ARG = 1 };

static void row_stats(const double *x, int64_t C, double eps, double *mean, double *rstd) {
    double s = 0.0;
    for (int64_t c = 0; c < C; ++c) s += x[c];
    const double mu = s / (double)C;
    double v = 0.0;
    for (int64_t c = 0; c < C; ++c) v += (x[c] - mu) * (x[c] - mu);
    v /= (double)C;
    *mean = mu;
    *rstd = 1.0 / sqrt(v + eps);
}

/* y, mean, rstd from x [R][C], w [C], b [C] (w or b NULL: 1 or 0) */
int ln_oracle_fwd(int64_t R, int64_t C, double eps, const double *x, const double *w,
                  const double *b, double *y, double *mean, double *rstd) {
    if (R < 0 || C <= 0 || eps < 0.0 || (R > 0 && (!x || !y))) return LN_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < R; ++r) {
        const double *xr = x + r * C;
        double mu, rs;
        row_stats(xr, C, eps, &mu, &rs);
        if (mean) mean[r] = mu;
        if (rstd) rstd[r] = rs;
        for (int64_t c = 0; c < C; ++c) {
            const double xh = (xr[c] - mu) * rs;
            y[r * C + c] = xh * (w ? w[c] : 1.0) + (b ? b[c] : 0.0);
        }
    }
    return LN_OK;
}

/* dx [R][C], dw [C], db [C] (dw, db may be NULL) from x, w, dy */
int ln_oracle_bwd(int64_t R, int64_t C, double eps, const double *x, const double *w,
                  const double *dy, double *dx, double *dw, double *db) {
    if (R < 0 || C <= 0 || eps < 0.0 || (R > 0 && (!x || !dy || !dx))) return LN_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < R; ++r) {
        const double *xr = x + r * C, *gr = dy + r * C;
        double mu, rs;
        row_stats(xr, C, eps, &mu, &rs);
        double sg = 0.0, sgx = 0.0;
        for (int64_t c = 0; c < C; ++c) {
            const double g = gr[c] * (w ? w[c] : 1.0);
            sg += g;
            sgx += g * (xr[c] - mu) * rs;
        }
        sg /= (double)C;
        sgx /= (double)C;
        for (int64_t c = 0; c < C; ++c) {
            const double g = gr[c] * (w ? w[c] : 1.0);
            const double xh = (xr[c] - mu) * rs;
            dx[r * C + c] = rs * (g - sg - xh * sgx);
        }
    }
    if (dw || db) {
        for (int64_t c = 0; c < C; ++c) {
            if (dw) dw[c] = 0.0;
            if (db) db[c] = 0.0;
        }
        for (int64_t r = 0; r < R; ++r) {
            const double *xr = x + r * C, *gr = dy + r * C;
            double mu, rs;
            row_stats(xr, C, eps, &mu, &rs);
            for (int64_t c = 0; c < C; ++c) {
                if (dw) dw[c] += gr[c] * (xr[c] - mu) * rs;
                if (db) db[c] += gr[c];
            }
        }
    }
    return LN_OK;
}
