/*
 * oracle_deep.c -- fp64 reference for mini-batch SGD on a d-h-...-h-1 ReLU/MSE
 * network: L hidden layers of width h, one output, no biases.
 *
 * TEST INFRASTRUCTURE ONLY, like oracle.c: linked only by tests, by the
 * package smoke check and by the CPU-baseline leg of the benchmark. The HIP
 * path never calls it, includes it or shares code with it, and this file
 * shares no code with oracle.c (the two are checked against each other at
 * L = 1).
 *
 * The paper trains a single hidden layer (Sec. III) and names deeper networks
 * as future work (Sec. VII.B). This is the chain rule of its equations applied
 * layer by layer, with the layer index of eq. (9):
 *   H_0 = X;  Z_l = H_{l-1} W_l,  H_l = ReLU(Z_l),  l = 1..L       eqs. (11)-(12)
 *   Ypred = H_L w_o                                                 eq. (13)
 *   L = (1/n_b) sum_i (Ypred_i - Y_i)^2                             eq. (14)
 *   dZ_o = (2/n_b)(Ypred - Y),  dw_o = H_L^T dZ_o                   eqs. (15)-(16)
 *   dH_L = dZ_o w_o^T
 *   dZ_l = dH_l (.) ReLU'(Z_l),  dW_l = H_{l-1}^T dZ_l              eqs. (17)-(18)
 *   dH_{l-1} = dZ_l W_l^T                                           (l >= 2)
 *   W_l <- W_l - alpha dW_l, w_o <- w_o - alpha dw_o, after every
 *   gradient is formed                                              eq. (19)
 * With L = 1 this is the network of oracle.c (W_1 = W1, w_o = W2). The
 * readings of oracle.c carry over: n_b is the row count of the batch, the last
 * batch keeps its remainder, ReLU'(0) = 0.
 *
 * Parameter layout, one flat array: W_1 [d x h] row-major (rows = inputs),
 * then W_2 ... W_L, each [h x h] row-major (rows = units of the layer below),
 * then w_o [h].
 *
 * Arithmetic: fp64 in the plain loop order written below (rows in batch
 * order; for each row the forward layer by layer, then the backward from the
 * output down), no blocking or reordering.
 *
 * Return codes: 0 success, -1 bad argument, -2 out of host memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ODP_OK 0
#define ODP_EINVAL -1
#define ODP_ENOMEM -2

int64_t oracle_deep_param_count(int32_t d, int32_t h, int32_t L) {
    if (d <= 0 || h <= 0 || L <= 0) return -1;
    return (int64_t)d * h + (int64_t)(L - 1) * h * h + h;
}

/* offset of W_l (l = 1..L) and of w_o (l = L + 1) in the flat array */
static int64_t layer_off(int32_t d, int32_t h, int32_t l) {
    if (l == 1) return 0;
    return (int64_t)d * h + (int64_t)(l - 2) * h * h;
}

static int64_t row_at(const int32_t *idx, int64_t t) { return idx ? (int64_t)idx[t] : t; }

/* Per-row scratch: the input of every layer (H_0 .. H_L) and every Z_l. */
typedef struct {
    double *hin;   /* [(L + 1) x w], w = max(d, h): hin[l] = H_l of the row */
    double *z;     /* [L x h] */
    double *dh;    /* [w] */
    double *dhn;   /* [w] */
    int32_t w;
} Rowbuf;

static int rowbuf_alloc(Rowbuf *b, int32_t d, int32_t h, int32_t L) {
    b->w = d > h ? d : h;
    b->hin = (double *)malloc(sizeof(double) * (size_t)(L + 1) * (size_t)b->w);
    b->z = (double *)malloc(sizeof(double) * (size_t)L * (size_t)h);
    b->dh = (double *)malloc(sizeof(double) * (size_t)b->w);
    b->dhn = (double *)malloc(sizeof(double) * (size_t)b->w);
    return b->hin && b->z && b->dh && b->dhn;
}

static void rowbuf_free(Rowbuf *b) {
    free(b->hin); free(b->z); free(b->dh); free(b->dhn);
}

/* Forward of one row, eqs. (11)-(13) per layer. Keeps H_l and Z_l in b and
 * returns Ypred. When margin != NULL, lowers *margin to the smallest
 * |Z_lj| / sum_k |H_{l-1,k} W_l,kj| seen (the relative size of a pre-activation
 * against the magnitude of its terms; 1 when that magnitude is 0). */
static double row_forward(const float *x, int32_t d, int32_t h, int32_t L, const double *P,
                          Rowbuf *b, double *margin) {
    for (int32_t k = 0; k < d; ++k) b->hin[k] = (double)x[k];
    for (int32_t l = 1; l <= L; ++l) {
        const int32_t K = l == 1 ? d : h;
        const double *W = P + layer_off(d, h, l);
        const double *hp = b->hin + (size_t)(l - 1) * b->w;
        double *hn = b->hin + (size_t)l * b->w;
        double *z = b->z + (size_t)(l - 1) * h;
        for (int32_t j = 0; j < h; ++j) {
            double acc = 0.0, mag = 0.0;
            for (int32_t k = 0; k < K; ++k) {
                double p = hp[k] * W[(int64_t)k * h + j];
                acc += p;
                mag += fabs(p);
            }
            z[j] = acc;
            hn[j] = acc > 0.0 ? acc : 0.0;                       /* eq. (12) */
            if (margin) {
                double m = mag > 0.0 ? fabs(acc) / mag : 1.0;
                if (m < *margin) *margin = m;
            }
        }
    }
    const double *wo = P + layer_off(d, h, L + 1);
    const double *hL = b->hin + (size_t)L * b->w;
    double y = 0.0;
    for (int32_t j = 0; j < h; ++j) y += hL[j] * wo[j];          /* eq. (13) */
    return y;
}

int oracle_deep_forward(const float *X, int64_t rows_X, const int32_t *idx, int64_t nb,
                        int32_t d, int32_t h, int32_t L, const double *P, double *ypred) {
    if (!X || !P || !ypred || d <= 0 || h <= 0 || L <= 0 || nb < 0 || rows_X < 0)
        return ODP_EINVAL;
    for (int64_t t = 0; t < nb; ++t) {
        int64_t r = row_at(idx, t);
        if (r < 0 || r >= rows_X) return ODP_EINVAL;
    }
    Rowbuf b;
    if (!rowbuf_alloc(&b, d, h, L)) { rowbuf_free(&b); return ODP_ENOMEM; }
    for (int64_t t = 0; t < nb; ++t)
        ypred[t] = row_forward(X + row_at(idx, t) * (int64_t)d, d, h, L, P, &b, NULL);
    rowbuf_free(&b);
    return ODP_OK;
}

/* Gradients of the batch MSE at the given parameters (eqs. 14-18 per layer),
 * summed over the rows in batch order. dP has the layout of P. *loss = L;
 * *margin (nullable) = the smallest relative pre-activation of the batch. */
int oracle_deep_grad(const float *X, const float *Y, int64_t rows_X, const int32_t *idx,
                     int64_t nb, int32_t d, int32_t h, int32_t L, const double *P, double *dP,
                     double *loss, double *margin) {
    if (!X || !Y || !P || !dP || d <= 0 || h <= 0 || L <= 0 || nb <= 0 || rows_X < 0)
        return ODP_EINVAL;
    for (int64_t t = 0; t < nb; ++t) {
        int64_t r = row_at(idx, t);
        if (r < 0 || r >= rows_X) return ODP_EINVAL;
    }
    const int64_t np = oracle_deep_param_count(d, h, L);
    Rowbuf b;
    if (!rowbuf_alloc(&b, d, h, L)) { rowbuf_free(&b); return ODP_ENOMEM; }
    memset(dP, 0, sizeof(double) * (size_t)np);
    if (margin) *margin = 1.0;
    const double scale = 2.0 / (double)nb;                      /* eq. (15), n = batch rows */
    const double *wo = P + layer_off(d, h, L + 1);
    double *dwo = dP + layer_off(d, h, L + 1);
    double sse = 0.0;
    for (int64_t t = 0; t < nb; ++t) {
        const int64_t r = row_at(idx, t);
        const double y = row_forward(X + r * (int64_t)d, d, h, L, P, &b, margin);
        const double res = y - (double)Y[r];
        sse += res * res;
        const double g = scale * res;
        /* output layer: dw_o = H_L^T dZ_o, dH_L = dZ_o w_o^T */
        const double *hL = b.hin + (size_t)L * b.w;
        for (int32_t j = 0; j < h; ++j) {
            dwo[j] += hL[j] * g;
            b.dh[j] = g * wo[j];
        }
        /* hidden layers, from the top down */
        for (int32_t l = L; l >= 1; --l) {
            const int32_t K = l == 1 ? d : h;
            const double *W = P + layer_off(d, h, l);
            double *dW = dP + layer_off(d, h, l);
            const double *hp = b.hin + (size_t)(l - 1) * b.w;
            const double *z = b.z + (size_t)(l - 1) * h;
            for (int32_t j = 0; j < h; ++j)                        /* dZ_l, eq. (17) */
                b.dh[j] = z[j] > 0.0 ? b.dh[j] : 0.0;
            for (int32_t k = 0; k < K; ++k)                        /* dW_l, eq. (18) */
                for (int32_t j = 0; j < h; ++j) dW[(int64_t)k * h + j] += hp[k] * b.dh[j];
            if (l > 1) {                                           /* dH_{l-1} = dZ_l W_l^T */
                for (int32_t k = 0; k < K; ++k) {
                    double acc = 0.0;
                    for (int32_t j = 0; j < h; ++j) acc += b.dh[j] * W[(int64_t)k * h + j];
                    b.dhn[k] = acc;
                }
                memcpy(b.dh, b.dhn, sizeof(double) * (size_t)K);
            }
        }
    }
    rowbuf_free(&b);
    if (loss) *loss = sse / (double)nb;
    return ODP_OK;
}

/* Mini-batch SGD over epochs (eq. 19 on every layer), the schedule of
 * oracle.c's oracle_train: epoch e visits perm[e*n ..] (identity when NULL) in
 * ceil(n/batch) steps, the last taking the remainder; stops after max_steps
 * steps when max_steps >= 0. step_loss[s] = batch loss before step s's update;
 * epoch_loss[e] = sum of the epoch's squared residuals / n. P is updated in
 * place. */
int oracle_deep_train(const float *X, const float *Y, int64_t n, int32_t d, int32_t h, int32_t L,
                      double *P, int64_t batch, double lr, int32_t epochs, const int32_t *perm,
                      int64_t max_steps, double *step_loss, double *epoch_loss,
                      int64_t *steps_done) {
    if (!X || !Y || !P || n <= 0 || d <= 0 || h <= 0 || L <= 0 || batch <= 0 || epochs < 0)
        return ODP_EINVAL;
    if (perm) {
        for (int64_t i = 0; i < (int64_t)epochs * n; ++i)
            if (perm[i] < 0 || perm[i] >= n) return ODP_EINVAL;
    }
    const int64_t np = oracle_deep_param_count(d, h, L);
    double *dP = (double *)malloc(sizeof(double) * (size_t)np);
    int32_t *ident = NULL;
    if (!dP) return ODP_ENOMEM;
    if (!perm) {
        ident = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        if (!ident) { free(dP); return ODP_ENOMEM; }
        for (int64_t i = 0; i < n; ++i) ident[i] = (int32_t)i;
    }
    int64_t steps = 0;
    int rc = ODP_OK;
    for (int32_t e = 0; e < epochs && rc == ODP_OK; ++e) {
        const int32_t *order = perm ? perm + (int64_t)e * n : ident;
        double epoch_sse = 0.0;
        if (epoch_loss) epoch_loss[e] = 0.0;
        for (int64_t s0 = 0; s0 < n; s0 += batch) {
            if (max_steps >= 0 && steps >= max_steps) break;
            const int64_t nb = n - s0 < batch ? n - s0 : batch;
            double Lb = 0.0;
            rc = oracle_deep_grad(X, Y, n, order + s0, nb, d, h, L, P, dP, &Lb, NULL);
            if (rc != ODP_OK) break;
            for (int64_t i = 0; i < np; ++i) P[i] -= lr * dP[i];   /* eq. (19) */
            if (step_loss) step_loss[steps] = Lb;
            epoch_sse += Lb * (double)nb;
            if (epoch_loss) epoch_loss[e] = epoch_sse / (double)n;
            ++steps;
        }
        if (max_steps >= 0 && steps >= max_steps) break;
    }
    free(dP);
    free(ident);
    if (steps_done) *steps_done = steps;
    return rc;
}
