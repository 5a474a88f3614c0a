// hostloop.hip -- the paper's two GPU strategies, rebuilt for gfx950 as
// host-driven step sequences so that they can be measured beside the fused
// trainer (the ablation of the paper's Sec. VI.B, Table I).
//
// Both compute one SGD step (eqs. 11-19) with every intermediate in device
// memory (the strategy workspace) and one kernel per operation, launched from
// the host for every step:
//
//   baseline (Sec. IV): every matrix product is a separate kernel with one
//     thread per output element in 16 x 16 blocks, operands read straight from
//     global memory (a transposed operand is read with a stride, eq. 20-22);
//     ReLU, the residual, the ReLU derivative and the update are separate
//     elementwise kernels.
//   optimized (Sec. V): products are LDS-tiled (16 x 16 tiles, two barriers per
//     K tile, Sec. V.A) in the form C = A Bt^T, so both operands are read
//     row-wise after an explicit transpose kernel (Sec. V.B); the ReLU is fused
//     into the product that makes Z1 (eq. 23, Sec. V.C) and the ReLU derivative
//     into the product that makes dZ1.
//
// Per step, in order: gather the batch rows; forward; residual and dZ2; loss;
// dW2; dZ1; dW1; update (or write the gradients). Each output element is
// computed by one thread in a fixed k order, and the loss by one workgroup in a
// fixed tree, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

constexpr int T16 = 16;

// ---------------------------------------------------------------------------
// Kernels shared by both strategies
// ---------------------------------------------------------------------------

// Xb[t][k] = X[r_t][k], Yb[t] = Y[r_t] with r_t = idx[off + t] (or off + t).
__global__ __launch_bounds__(256) void k_hl_gather(const float *__restrict__ X,
                                                   const float *__restrict__ Y, int64_t n_rows,
                                                   const int32_t *__restrict__ idx, int64_t off,
                                                   int64_t nb, float *__restrict__ Xb,
                                                   float *__restrict__ Yb, int32_t *err) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= nb * D_IN) return;
    const int64_t t = e / D_IN;
    const int k = (int)(e % D_IN);
    int64_t r = idx ? (int64_t)idx[off + t] : off + t;
    if (r < 0 || r >= n_rows) {
        __hip_atomic_store(err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r = 0;
    }
    Xb[e] = X[r * D_IN + k];
    if (k == 0) Yb[t] = Y ? Y[r] : 0.0f;
}

// r = Ypred - Y (eq. 14), dZ2 = (2/n_b) r (eq. 15), sq = r^2.
__global__ __launch_bounds__(256) void k_hl_residual(const float *__restrict__ yp,
                                                     const float *__restrict__ Yb, int64_t nb,
                                                     float scale, float *__restrict__ dz2,
                                                     float *__restrict__ sq) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= nb) return;
    const float r = yp[t] - Yb[t];
    dz2[t] = scale * r;
    sq[t] = r * r;
}

// Batch loss (eq. 14) from the squared residuals: one workgroup; thread i sums
// entries i, i + 256, ... in order, then a fixed binary tree over the threads.
__global__ __launch_bounds__(256) void k_hl_loss(const float *__restrict__ sq, int64_t nb,
                                                 ReduceArgs a) {
    __shared__ float part[256];
    const int i = threadIdx.x;
    float s = 0.0f;
    for (int64_t t = i; t < nb; t += 256) s += sq[t];
    part[i] = s;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (i < w) part[i] += part[i + w];
        __syncthreads();
    }
    if (i == 0) {
        const float sse = part[0];
        const float L = sse * a.inv_nb;
        flag_nonfinite(sse, &a.ctl->err);
        if (a.loss) a.loss[0] = L;
        if (a.step_loss) a.step_loss[a.step] = L;
        if (a.epoch_loss) {
            double acc = a.first_in_epoch ? 0.0 : a.ctl->epoch_sse;
            acc += (double)sse;
            a.ctl->epoch_sse = acc;
            a.epoch_loss[a.epoch] = (float)(acc * a.inv_n);
        }
    }
}

// Eq. 19 (sgd) or the gradient outputs: one thread per weight of [W1 | W2].
__global__ __launch_bounds__(256) void k_hl_apply(const float *__restrict__ dW1,
                                                  const float *__restrict__ dW2, int hidden,
                                                  ReduceArgs a) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int n1 = D_IN * hidden;
    if (t < n1) {
        if (a.sgd) a.W1[t] -= a.lr * dW1[t];
        else a.dW1[t] = dW1[t];
    } else if (t < n1 + hidden) {
        if (a.sgd) a.W2[t - n1] -= a.lr * dW2[t - n1];
        else a.dW2[t - n1] = dW2[t - n1];
    }
}

// ---------------------------------------------------------------------------
// Baseline strategy (Sec. IV)
// ---------------------------------------------------------------------------

// C[i][j] = sum_k A(i, k) B(k, j), A(i, k) = A[i sai + k sak], B(k, j) =
// B[k sbk + j sbj]; C row-major [M x N]. Thread (x, y) of block (bx, by)
// computes C[16 bx + y][16 by + x] from global memory alone (eq. 20).
__global__ __launch_bounds__(256) void k_gemm_naive(const float *__restrict__ A, int64_t sai,
                                                    int64_t sak, const float *__restrict__ B,
                                                    int64_t sbk, int64_t sbj,
                                                    float *__restrict__ C, int64_t M, int N,
                                                    int64_t K) {
    const int64_t i = (int64_t)blockIdx.x * T16 + threadIdx.y;
    const int j = blockIdx.y * T16 + threadIdx.x;
    if (i >= M || j >= N) return;
    float acc = 0.0f;
    for (int64_t k = 0; k < K; ++k) acc = fmaf(A[i * sai + k * sak], B[k * sbk + j * sbj], acc);
    C[i * N + j] = acc;
}

// H = ReLU(Z1) (eq. 12), a kernel of its own.
__global__ __launch_bounds__(256) void k_hl_relu(const float *__restrict__ Z, float *__restrict__ H,
                                                 int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e < n) H[e] = Z[e] > 0.0f ? Z[e] : 0.0f;
}

// dZ1 = G (.) ReLU'(Z1), ReLU'(z) = [z > 0] (eq. 17), a kernel of its own.
__global__ __launch_bounds__(256) void k_hl_relu_grad(const float *__restrict__ G,
                                                      const float *__restrict__ Z,
                                                      float *__restrict__ D, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e < n) D[e] = Z[e] > 0.0f ? G[e] : 0.0f;
}

// ---------------------------------------------------------------------------
// Optimized strategy (Sec. V)
// ---------------------------------------------------------------------------

// dst [cols x rows] = src [rows x cols]^T through a 16 x 17 LDS tile, so that
// both the reads and the writes are row-wise (Sec. V.B).
__global__ __launch_bounds__(256) void k_transpose(const float *__restrict__ src,
                                                   float *__restrict__ dst, int64_t rows,
                                                   int64_t cols) {
    __shared__ float tile[T16][T16 + 1];
    const int64_t r0 = (int64_t)blockIdx.x * T16, c0 = (int64_t)blockIdx.y * T16;
    const int x = threadIdx.x, y = threadIdx.y;
    if (r0 + y < rows && c0 + x < cols) tile[y][x] = src[(r0 + y) * cols + c0 + x];
    __syncthreads();
    if (c0 + y < cols && r0 + x < rows) dst[(c0 + y) * rows + r0 + x] = tile[x][y];
}

enum { EPI_NONE = 0, EPI_RELU = 1, EPI_MASK = 2 };

// C [M x N] = A [M x K] Bt [N x K]^T, both operands row-major and read row-wise
// through 16 x 16 LDS tiles (Sec. V.A); k ascending. Epilogue in registers:
// EPI_RELU applies eq. 12 (eq. 23's fusion), EPI_MASK keeps C where G > 0
// (eq. 17 with G = H, since H > 0 exactly where Z1 > 0).
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_tiled(const float *__restrict__ A,
                                                    const float *__restrict__ Bt,
                                                    float *__restrict__ C, int64_t M, int N,
                                                    int64_t K, const float *__restrict__ G) {
    __shared__ float As[T16][T16 + 1], Bs[T16][T16 + 1];
    const int x = threadIdx.x, y = threadIdx.y;
    const int64_t i0 = (int64_t)blockIdx.x * T16;
    const int j0 = blockIdx.y * T16;
    float acc = 0.0f;
    for (int64_t k0 = 0; k0 < K; k0 += T16) {
        As[y][x] = (i0 + y < M && k0 + x < K) ? A[(i0 + y) * K + k0 + x] : 0.0f;
        Bs[y][x] = (j0 + y < N && k0 + x < K) ? Bt[(int64_t)(j0 + y) * K + k0 + x] : 0.0f;
        __syncthreads();
        const int kn = K - k0 < T16 ? (int)(K - k0) : T16;
        for (int kk = 0; kk < kn; ++kk) acc = fmaf(As[y][kk], Bs[x][kk], acc);
        __syncthreads();
    }
    const int64_t i = i0 + y;
    const int j = j0 + x;
    if (i >= M || j >= N) return;
    float v = acc;
    if (EPI == EPI_RELU) v = v > 0.0f ? v : 0.0f;
    if (EPI == EPI_MASK) v = G[i * N + j] > 0.0f ? v : 0.0f;
    C[i * N + j] = v;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

// Strategy workspace, in floats: Xb, XbT [nb x 32] each; Yb, yp, dz2, sq [nb];
// Z1, H, HT, G, dZ1, dZ1T [nb x h] each; W1T, dW1 [32 h]; dW2 [h]. Every array
// starts on a 256-byte boundary.
struct HLBufs {
    float *Xb, *XbT, *Yb, *yp, *dz2, *sq, *Z1, *H, *HT, *G, *dZ1, *dZ1T, *W1T, *dW1, *dW2;
};

static size_t pad64(size_t n) { return (n + 63) / 64 * 64; }

size_t hostloop_workspace_floats(int hidden, int64_t max_batch) {
    const size_t nb = (size_t)max_batch, h = (size_t)hidden;
    return 2 * pad64(nb * D_IN) + 4 * pad64(nb) + 6 * pad64(nb * h) + 2 * pad64(D_IN * h) +
           pad64(h);
}

static HLBufs carve(const Ctx &c) {
    const size_t nb = (size_t)c.hl_max_batch, h = (size_t)c.hidden;
    float *p = c.hl_ws;
    auto take = [&](size_t n) {
        float *q = p;
        p += pad64(n);
        return q;
    };
    HLBufs b;
    b.Xb = take(nb * D_IN);
    b.XbT = take(nb * D_IN);
    b.Yb = take(nb);
    b.yp = take(nb);
    b.dz2 = take(nb);
    b.sq = take(nb);
    b.Z1 = take(nb * h);
    b.H = take(nb * h);
    b.HT = take(nb * h);
    b.G = take(nb * h);
    b.dZ1 = take(nb * h);
    b.dZ1T = take(nb * h);
    b.W1T = take(D_IN * h);
    b.dW1 = take(D_IN * h);
    b.dW2 = take(h);
    return b;
}

static unsigned blocks256(int64_t n) { return (unsigned)((n + 255) / 256); }
static unsigned tiles16(int64_t n) { return (unsigned)((n + T16 - 1) / T16); }

static hipError_t naive(const Ctx &c, const float *A, int64_t sai, int64_t sak, const float *B,
                        int64_t sbk, int64_t sbj, float *C, int64_t M, int N, int64_t K) {
    hipLaunchKernelGGL(k_gemm_naive, dim3(tiles16(M), tiles16(N)), dim3(T16, T16), 0, c.stream, A,
                       sai, sak, B, sbk, sbj, C, M, N, K);
    return hipGetLastError();
}

template <int EPI>
static hipError_t tiled(const Ctx &c, const float *A, const float *Bt, float *C, int64_t M, int N,
                        int64_t K, const float *G) {
    hipLaunchKernelGGL((k_gemm_tiled<EPI>), dim3(tiles16(M), tiles16(N)), dim3(T16, T16), 0,
                       c.stream, A, Bt, C, M, N, K, G);
    return hipGetLastError();
}

static hipError_t transpose(const Ctx &c, const float *src, float *dst, int64_t rows, int64_t cols) {
    hipLaunchKernelGGL(k_transpose, dim3(tiles16(rows), tiles16(cols)), dim3(T16, T16), 0, c.stream,
                       src, dst, rows, cols);
    return hipGetLastError();
}

#define HL_TRY(x)                          \
    do {                                   \
        hipError_t e_ = (x);               \
        if (e_ != hipSuccess) return e_;   \
    } while (0)

int hostloop_launches_per_step(int strategy) { return strategy == MLP_STRATEGY_BASELINE ? 11 : 13; }

hipError_t hostloop_step(const Ctx &c, const float *X, int64_t n_rows, const float *Y,
                         const int32_t *idx, int64_t idx_off, int64_t nb, const ReduceArgs &a) {
    const HLBufs b = carve(c);
    const int h = c.hidden;
    const float scale = 2.0f / (float)nb;   // eq. 15
    const int64_t nh = nb * h;
    hipLaunchKernelGGL(k_hl_gather, dim3(blocks256(nb * D_IN)), dim3(256), 0, c.stream, X, Y,
                       n_rows, idx, idx_off, nb, b.Xb, b.Yb, &c.ctl->err);
    HL_TRY(hipGetLastError());
    if (c.strategy == MLP_STRATEGY_BASELINE) {
        // eq. 11: Z1 = Xb W1; eq. 12: H = ReLU(Z1); eq. 13: Ypred = H W2
        HL_TRY(naive(c, b.Xb, D_IN, 1, c.W1, h, 1, b.Z1, nb, h, D_IN));
        hipLaunchKernelGGL(k_hl_relu, dim3(blocks256(nh)), dim3(256), 0, c.stream, b.Z1, b.H, nh);
        HL_TRY(hipGetLastError());
        HL_TRY(naive(c, b.H, h, 1, c.W2, 1, 1, b.yp, nb, 1, h));
    } else {
        // W1^T once per step (the weights change every step), then eq. 11 with
        // eq. 12 fused; Ypred = H W2 with W2 read as a [1 x h] row
        HL_TRY(transpose(c, c.W1, b.W1T, D_IN, h));
        HL_TRY(tiled<EPI_RELU>(c, b.Xb, b.W1T, b.H, nb, h, D_IN, nullptr));
        HL_TRY(tiled<EPI_NONE>(c, b.H, c.W2, b.yp, nb, 1, h, nullptr));
    }
    hipLaunchKernelGGL(k_hl_residual, dim3(blocks256(nb)), dim3(256), 0, c.stream, b.yp, b.Yb, nb,
                       scale, b.dz2, b.sq);
    HL_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_hl_loss, dim3(1), dim3(256), 0, c.stream, b.sq, nb, a);
    HL_TRY(hipGetLastError());
    if (c.strategy == MLP_STRATEGY_BASELINE) {
        // eq. 16: dW2 = H^T dZ2 (H read by column); eq. 17: dZ1 = (dZ2 W2^T) (.)
        // ReLU'(Z1); eq. 18: dW1 = Xb^T dZ1 (Xb read by column)
        HL_TRY(naive(c, b.H, 1, h, b.dz2, 1, 1, b.dW2, h, 1, nb));
        HL_TRY(naive(c, b.dz2, 1, 1, c.W2, 1, 1, b.G, nb, h, 1));
        hipLaunchKernelGGL(k_hl_relu_grad, dim3(blocks256(nh)), dim3(256), 0, c.stream, b.G, b.Z1,
                           b.dZ1, nh);
        HL_TRY(hipGetLastError());
        HL_TRY(naive(c, b.Xb, 1, D_IN, b.dZ1, h, 1, b.dW1, D_IN, h, nb));
    } else {
        // eq. 16 on H^T; eq. 17 as a K = 1 product with the derivative fused;
        // eq. 18 on Xb^T and dZ1^T
        HL_TRY(transpose(c, b.H, b.HT, nb, h));
        HL_TRY(tiled<EPI_NONE>(c, b.HT, b.dz2, b.dW2, h, 1, nb, nullptr));
        HL_TRY(tiled<EPI_MASK>(c, b.dz2, c.W2, b.dZ1, nb, h, 1, b.H));
        HL_TRY(transpose(c, b.Xb, b.XbT, nb, D_IN));
        HL_TRY(transpose(c, b.dZ1, b.dZ1T, nb, h));
        HL_TRY(tiled<EPI_NONE>(c, b.XbT, b.dZ1T, b.dW1, D_IN, h, nb, nullptr));
    }
    // eq. 19, or the gradient outputs
    hipLaunchKernelGGL(k_hl_apply, dim3(blocks256((int64_t)(D_IN + 1) * h)), dim3(256), 0, c.stream,
                       b.dW1, b.dW2, h, a);
    return hipGetLastError();
}

}  // namespace mlp
