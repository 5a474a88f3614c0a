/*
 * oracle_mt.c -- the fp64 reference of oracle.c run on several host cores.
 *
 * TEST INFRASTRUCTURE ONLY. Linked by tests and by the CPU-baseline leg of the
 * benchmark; the HIP training path never calls it, includes it or shares code
 * with it. It shares no code with oracle.c either: the per-row loops below are
 * written out again, in the same equation order.
 *
 * What it computes is the mini-batch SGD of paper Sec. III eqs. (11)-(19) with
 * the readings of oracle.c (n in eqs. 14-15 = rows of the current batch; the
 * last batch keeps its remainder; ReLU'(0) = 0; both gradients from the
 * pre-update weights; every step on the current weights). The one difference
 * is the order of the batch sums: every batch is cut into NCHUNK contiguous
 * row ranges (chunk c holds batch rows [c*nb/NCHUNK, (c+1)*nb/NCHUNK)); each
 * chunk sums its rows in batch order into its own partial (dW1, dW2, squared
 * residuals), and the partials are added in chunk order. The partition does
 * not depend on the number of threads, so the result does not either; against
 * oracle.c it differs only by the rounding of the reassociated sums.
 *
 * The forward pass (eqs. 11-13) has no sum across rows: oracle_mt_forward
 * returns exactly what oracle_forward returns, row by row, on any number of
 * threads.
 *
 * Arithmetic: fp32 inputs promoted to fp64; every sum and product in fp64.
 * Return codes: 0 success, -1 bad argument, -2 out of host memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MT_OK 0
#define MT_EINVAL -1
#define MT_ENOMEM -2
#define NCHUNK 64

static int64_t mt_row(const int32_t *idx, int64_t t) { return idx ? (int64_t)idx[t] : t; }

/* Number of threads an OpenMP region of this library uses (1 without OpenMP). */
int oracle_mt_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for the following calls (n >= 1); returns the previous count. */
int oracle_mt_set_threads(int n) {
    const int prev = oracle_mt_threads();
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
    return prev;
}

/* Ypred for rows idx[0..nb) (idx NULL: rows 0..nb-1), eqs. (11)-(13). */
int oracle_mt_forward(const float *X, int64_t rows_X, const int32_t *idx, int64_t nb, int32_t d,
                      int32_t h, const double *W1, const double *W2, double *ypred) {
    if (!X || !W1 || !W2 || !ypred || d <= 0 || h <= 0 || nb < 0 || rows_X < 0) return MT_EINVAL;
    for (int64_t t = 0; t < nb; ++t) {
        const int64_t r = mt_row(idx, t);
        if (r < 0 || r >= rows_X) return MT_EINVAL;
    }
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < nb; ++t) {
        const float *x = X + mt_row(idx, t) * (int64_t)d;
        double y = 0.0;
        for (int32_t j = 0; j < h; ++j) {
            double z = 0.0;
            for (int32_t k = 0; k < d; ++k) z += (double)x[k] * W1[(int64_t)k * h + j];   /* eq. (11) */
            y += (z > 0.0 ? z : 0.0) * W2[j];                                           /* eqs. (12)-(13) */
        }
        ypred[t] = y;
    }
    return MT_OK;
}

/* One chunk of a batch: rows t in [t0, t1) of the batch, in order, into the
 * chunk's partials p1 [d x h], p2 [h] and *sse. scale = 2 / n_b of the whole
 * batch (eq. 15). */
static void chunk_grad(const float *X, const float *Y, const int32_t *idx, int64_t t0, int64_t t1,
                       int32_t d, int32_t h, const double *W1, const double *W2, double scale,
                       double *z, double *p1, double *p2, double *sse) {
    memset(p1, 0, sizeof(double) * (size_t)d * (size_t)h);
    memset(p2, 0, sizeof(double) * (size_t)h);
    double s = 0.0;
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t r = mt_row(idx, t);
        const float *x = X + r * (int64_t)d;
        double y = 0.0;
        for (int32_t j = 0; j < h; ++j) {
            double acc = 0.0;
            for (int32_t k = 0; k < d; ++k) acc += (double)x[k] * W1[(int64_t)k * h + j];   /* eq. (11) */
            z[j] = acc;
            y += (acc > 0.0 ? acc : 0.0) * W2[j];                                          /* eqs. (12)-(13) */
        }
        const double res = y - (double)Y[r];                                              /* eq. (14) */
        s += res * res;
        const double g = scale * res;                                                     /* eq. (15) */
        for (int32_t j = 0; j < h; ++j) {
            p2[j] += (z[j] > 0.0 ? z[j] : 0.0) * g;                                       /* eq. (16) */
            const double dz1 = z[j] > 0.0 ? g * W2[j] : 0.0;                              /* eq. (17) */
            for (int32_t k = 0; k < d; ++k) p1[(int64_t)k * h + j] += (double)x[k] * dz1;  /* eq. (18) */
        }
    }
    *sse = s;
}

/* Gradient of one batch of nb rows from NCHUNK chunk partials summed in chunk
 * order. part: NCHUNK * (d*h + h + 1) doubles of scratch; zs: NCHUNK * h. */
static void batch_grad(const float *X, const float *Y, const int32_t *idx, int64_t nb, int32_t d,
                       int32_t h, const double *W1, const double *W2, double *part, double *zs,
                       double *dW1, double *dW2, double *sse_out) {
    const size_t n1 = (size_t)d * (size_t)h, stride = n1 + (size_t)h + 1;
    const double scale = 2.0 / (double)nb;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < NCHUNK; ++c) {
        double *p = part + (size_t)c * stride;
        chunk_grad(X, Y, idx, (int64_t)c * nb / NCHUNK, (int64_t)(c + 1) * nb / NCHUNK, d, h, W1, W2,
                   scale, zs + (size_t)c * (size_t)h, p, p + n1, p + n1 + h);
    }
    memset(dW1, 0, sizeof(double) * n1);
    memset(dW2, 0, sizeof(double) * (size_t)h);
    double sse = 0.0;
    for (int c = 0; c < NCHUNK; ++c) {
        const double *p = part + (size_t)c * stride;
        for (size_t i = 0; i < n1; ++i) dW1[i] += p[i];
        for (int32_t j = 0; j < h; ++j) dW2[j] += p[n1 + j];
        sse += p[n1 + h];
    }
    *sse_out = sse;
}

/* Gradients of the batch MSE at the given weights (eqs. 14-18), chunked. */
int oracle_mt_grad(const float *X, const float *Y, int64_t rows_X, const int32_t *idx, int64_t nb,
                   int32_t d, int32_t h, const double *W1, const double *W2, double *dW1,
                   double *dW2, double *loss) {
    if (!X || !Y || !W1 || !W2 || !dW1 || !dW2 || d <= 0 || h <= 0 || nb <= 0 || rows_X < 0)
        return MT_EINVAL;
    for (int64_t t = 0; t < nb; ++t) {
        const int64_t r = mt_row(idx, t);
        if (r < 0 || r >= rows_X) return MT_EINVAL;
    }
    const size_t stride = (size_t)d * (size_t)h + (size_t)h + 1;
    double *part = (double *)malloc(sizeof(double) * stride * NCHUNK);
    double *zs = (double *)malloc(sizeof(double) * (size_t)h * NCHUNK);
    if (!part || !zs) { free(part); free(zs); return MT_ENOMEM; }
    double sse = 0.0;
    batch_grad(X, Y, idx, nb, d, h, W1, W2, part, zs, dW1, dW2, &sse);
    free(part); free(zs);
    if (loss) *loss = sse / (double)nb;
    return MT_OK;
}

/* Mini-batch SGD over epochs (eq. 19 after every batch), the loop of
 * oracle_train with chunked batch gradients. Same arguments and outputs. */
int oracle_mt_train(const float *X, const float *Y, int64_t n, int32_t d, int32_t h, double *W1,
                    double *W2, int64_t batch, double lr, int32_t epochs, const int32_t *perm,
                    int64_t max_steps, double *step_loss, double *epoch_loss, int64_t *steps_done) {
    if (!X || !Y || !W1 || !W2 || n <= 0 || d <= 0 || h <= 0 || batch <= 0 || epochs < 0)
        return MT_EINVAL;
    if (perm)
        for (int64_t i = 0; i < (int64_t)epochs * n; ++i)
            if (perm[i] < 0 || perm[i] >= n) return MT_EINVAL;
    const size_t n1 = (size_t)d * (size_t)h, stride = n1 + (size_t)h + 1;
    double *dW1 = (double *)malloc(sizeof(double) * n1);
    double *dW2 = (double *)malloc(sizeof(double) * (size_t)h);
    double *part = (double *)malloc(sizeof(double) * stride * NCHUNK);
    double *zs = (double *)malloc(sizeof(double) * (size_t)h * NCHUNK);
    if (!dW1 || !dW2 || !part || !zs) {
        free(dW1); free(dW2); free(part); free(zs);
        return MT_ENOMEM;
    }
    int64_t steps = 0;
    for (int32_t e = 0; e < epochs; ++e) {
        double epoch_sse = 0.0;
        if (epoch_loss) epoch_loss[e] = 0.0;
        for (int64_t s0 = 0; s0 < n; s0 += batch) {
            if (max_steps >= 0 && steps >= max_steps) break;
            const int64_t nb = (n - s0 < batch) ? (n - s0) : batch;
            const int32_t *rows = perm ? perm + (int64_t)e * n + s0 : NULL;
            double sse = 0.0;
            if (rows) {
                batch_grad(X, Y, rows, nb, d, h, W1, W2, part, zs, dW1, dW2, &sse);
            } else {
                /* identity order: rows s0 .. s0 + nb - 1 */
                batch_grad(X + s0 * (int64_t)d, Y + s0, NULL, nb, d, h, W1, W2, part, zs, dW1,
                           dW2, &sse);
            }
            const double L = sse / (double)nb;                                           /* eq. (14) */
            for (size_t i = 0; i < n1; ++i) W1[i] -= lr * dW1[i];                         /* eq. (19) */
            for (int32_t j = 0; j < h; ++j) W2[j] -= lr * dW2[j];
            if (step_loss) step_loss[steps] = L;
            epoch_sse += sse;
            if (epoch_loss) epoch_loss[e] = epoch_sse / (double)n;
            ++steps;
        }
        if (max_steps >= 0 && steps >= max_steps) break;
    }
    free(dW1); free(dW2); free(part); free(zs);
    if (steps_done) *steps_done = steps;
    return MT_OK;
}
