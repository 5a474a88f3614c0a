/*
 * oracle.c -- fp64 reference for mini-batch SGD on a d-h-1 ReLU/MSE network
 * with no biases.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the correctness oracle. It is linked
 * only by tests, by the package smoke check and by the CPU-baseline leg of the
 * benchmark. The HIP training path never calls it, includes it or shares code
 * with it.
 *
 * What it computes (paper Sec. II.A eqs. (1)-(9), restated in Sec. III
 * eqs. (11)-(19)), for one mini-batch of n_b rows:
 *   Z1 = X W1, H = ReLU(Z1), Ypred = H W2                       eqs. (11)-(13)
 *   L  = (1/n_b) sum_i (Ypred_i - Y_i)^2                         eq. (14)
 *   dZ2 = (2/n_b)(Ypred - Y)                                     eq. (15)
 *   dW2 = H^T dZ2                                                eq. (16)
 *   dZ1 = (dZ2 W2^T) (.) ReLU'(Z1), ReLU'(x) = [x > 0]           eq. (17)
 *   dW1 = X^T dZ1                                                eq. (18)
 *   W  <- W - alpha dW   for both layers, after both gradients   eq. (19)
 * Readings where the paper is silent or ambiguous:
 *   - n in eqs. (14)-(15) is the row count of the current mini-batch;
 *   - the last batch of an epoch keeps its remainder rows (no drop) and
 *     scales by its own row count;
 *   - ReLU(0) = 0 and ReLU'(0) = 0 (strict x > 0, Sec. III.C);
 *   - both gradients use the weights from before the update;
 *   - every step uses the current weights (a transposed copy, Sec. V.B, is a
 *     layout choice and never a stale operand).
 *
 * Arithmetic: inputs arrive as fp32 (the values the device sees) and are
 * promoted; every sum and product is fp64, in the plain loop order written
 * below (rows in batch order, k ascending, j ascending). No blocking, no
 * reordering, no fused kernels.
 *
 * Layouts: X [rows x d] row-major, Y [rows], W1 [d x h] row-major with rows =
 * inputs (paper layout), W2 [h], perm [epochs x n] int32.
 *
 * Return codes: 0 success, -1 bad argument (null pointer, non-positive size,
 * row index out of range), -2 out of host memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL -1
#define ORC_ENOMEM -2

static int64_t row_of(const int32_t *idx, int64_t t) { return idx ? (int64_t)idx[t] : t; }

/* Check that every referenced row lies in [0, rows_X). */
static int rows_ok(const int32_t *idx, int64_t nb, int64_t rows_X) {
    for (int64_t t = 0; t < nb; ++t) {
        int64_t r = row_of(idx, t);
        if (r < 0 || r >= rows_X) return 0;
    }
    return 1;
}

/* Forward pass only, eqs. (11)-(13): ypred[t] for rows idx[0..nb)
 * (idx == NULL selects rows 0..nb-1). */
int oracle_forward(const float *X, int64_t rows_X, const int32_t *idx, int64_t nb,
                   int32_t d, int32_t h, const double *W1, const double *W2,
                   double *ypred) {
    if (!X || !W1 || !W2 || !ypred || d <= 0 || h <= 0 || nb < 0 || rows_X < 0)
        return ORC_EINVAL;
    if (!rows_ok(idx, nb, rows_X)) return ORC_EINVAL;
    for (int64_t t = 0; t < nb; ++t) {
        const float *x = X + row_of(idx, t) * (int64_t)d;
        double y = 0.0;
        for (int32_t j = 0; j < h; ++j) {
            double z = 0.0;
            for (int32_t k = 0; k < d; ++k) z += (double)x[k] * W1[(int64_t)k * h + j];
            double hj = z > 0.0 ? z : 0.0;                 /* eq. (12) */
            y += hj * W2[j];                               /* eq. (13) */
        }
        ypred[t] = y;
    }
    return ORC_OK;
}

/* Gradients of the batch MSE at the given weights, eqs. (14)-(18).
 * Outputs dW1 [d x h], dW2 [h], *loss = L (eq. 14). Optional outputs:
 *   z_out   [nb x h]: the pre-activations Z1 (eq. 11);
 *   zabs_out[nb x h]: sum_k |X_ik W1_kj|, the magnitude scale of each Z1 entry,
 *                     used by tests to find entries whose sign fp32 cannot
 *                     resolve. */
int oracle_grad(const float *X, const float *Y, int64_t rows_X, const int32_t *idx,
                int64_t nb, int32_t d, int32_t h, const double *W1, const double *W2,
                double *dW1, double *dW2, double *loss, double *z_out, double *zabs_out) {
    if (!X || !Y || !W1 || !W2 || !dW1 || !dW2 || d <= 0 || h <= 0 || nb <= 0 || rows_X < 0)
        return ORC_EINVAL;
    if (!rows_ok(idx, nb, rows_X)) return ORC_EINVAL;
    double *z = (double *)malloc(sizeof(double) * (size_t)h);
    if (!z) return ORC_ENOMEM;
    memset(dW1, 0, sizeof(double) * (size_t)d * (size_t)h);
    memset(dW2, 0, sizeof(double) * (size_t)h);
    double sse = 0.0;
    const double scale = 2.0 / (double)nb;                 /* eq. (15), n = batch rows */
    for (int64_t t = 0; t < nb; ++t) {
        const int64_t r = row_of(idx, t);
        const float *x = X + r * (int64_t)d;
        /* forward, eqs. (11)-(13) */
        double y = 0.0;
        for (int32_t j = 0; j < h; ++j) {
            double acc = 0.0, mag = 0.0;
            for (int32_t k = 0; k < d; ++k) {
                double p = (double)x[k] * W1[(int64_t)k * h + j];
                acc += p;
                mag += fabs(p);
            }
            z[j] = acc;
            if (z_out) z_out[t * h + j] = acc;
            if (zabs_out) zabs_out[t * h + j] = mag;
            y += (acc > 0.0 ? acc : 0.0) * W2[j];
        }
        /* residual, loss and output gradient, eqs. (14)-(15) */
        double res = y - (double)Y[r];
        sse += res * res;
        double g = scale * res;
        /* eqs. (16)-(18): dW2 += H^T g, dZ1 = g W2 (.) [Z1 > 0], dW1 += X^T dZ1 */
        for (int32_t j = 0; j < h; ++j) {
            double hj = z[j] > 0.0 ? z[j] : 0.0;
            dW2[j] += hj * g;
            double dz1 = z[j] > 0.0 ? g * W2[j] : 0.0;
            for (int32_t k = 0; k < d; ++k) dW1[(int64_t)k * h + j] += (double)x[k] * dz1;
        }
    }
    free(z);
    if (loss) *loss = sse / (double)nb;
    return ORC_OK;
}

/* Mini-batch SGD over epochs (Sec. II.A, Sec. III.A, eq. (19)).
 * Epoch e visits rows perm[e*n + 0 .. n-1] in order (perm == NULL: 0..n-1),
 * in ceil(n/batch) batches; the last keeps the remainder. W1/W2 are updated in
 * place (fp64). Stops after max_steps steps when max_steps >= 0.
 * step_loss[s] = batch loss of step s before its update (eq. 14);
 * epoch_loss[e] = (sum over the epoch's batches of their squared residuals) / n.
 * *steps_done receives the number of steps taken. */
int oracle_train(const float *X, const float *Y, int64_t n, int32_t d, int32_t h,
                 double *W1, double *W2, int64_t batch, double lr, int32_t epochs,
                 const int32_t *perm, int64_t max_steps, double *step_loss,
                 double *epoch_loss, int64_t *steps_done) {
    if (!X || !Y || !W1 || !W2 || n <= 0 || d <= 0 || h <= 0 || batch <= 0 || epochs < 0)
        return ORC_EINVAL;
    if (perm) {
        for (int64_t i = 0; i < (int64_t)epochs * n; ++i)
            if (perm[i] < 0 || perm[i] >= n) return ORC_EINVAL;
    }
    const size_t n1 = (size_t)d * (size_t)h;
    double *dW1 = (double *)malloc(sizeof(double) * n1);
    double *dW2 = (double *)malloc(sizeof(double) * (size_t)h);
    int32_t *ident = NULL;
    if (!dW1 || !dW2) { free(dW1); free(dW2); return ORC_ENOMEM; }
    if (!perm) {
        ident = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        if (!ident) { free(dW1); free(dW2); return ORC_ENOMEM; }
        for (int64_t i = 0; i < n; ++i) ident[i] = (int32_t)i;
    }
    int64_t steps = 0;
    int rc = ORC_OK;
    for (int32_t e = 0; e < epochs && rc == ORC_OK; ++e) {
        const int32_t *order = perm ? perm + (int64_t)e * n : ident;
        double epoch_sse = 0.0;
        if (epoch_loss) epoch_loss[e] = 0.0;
        for (int64_t s0 = 0; s0 < n; s0 += batch) {
            if (max_steps >= 0 && steps >= max_steps) break;
            int64_t nb = (n - s0 < batch) ? (n - s0) : batch;
            double L = 0.0;
            rc = oracle_grad(X, Y, n, order + s0, nb, d, h, W1, W2, dW1, dW2, &L, NULL, NULL);
            if (rc != ORC_OK) break;
            for (size_t i = 0; i < n1; ++i) W1[i] -= lr * dW1[i];          /* eq. (19) */
            for (int32_t j = 0; j < h; ++j) W2[j] -= lr * dW2[j];
            if (step_loss) step_loss[steps] = L;
            epoch_sse += L * (double)nb;
            if (epoch_loss) epoch_loss[e] = epoch_sse / (double)n;
            ++steps;
        }
        if (max_steps >= 0 && steps >= max_steps) break;
    }
    free(dW1); free(dW2); free(ident);
    if (steps_done) *steps_done = steps;
    return rc;
}
