// mlp.hip -- HIP (gfx950) implementation of the C ABI in include/mlp.h:
// fused mini-batch SGD for the d-h-1 ReLU/MSE network of the paper's
// Sec. III (eqs. 11-19), d = 32, no biases.
//
// Kernels in this file (the "tile" path):
//   k_tile<H>       one workgroup owns a contiguous slice of the batch; thread j
//                   owns hidden unit j. Rows are staged through LDS in groups of
//                   RG; Z1, the ReLU mask, H and dZ1 live only in registers
//                   (never in HBM). It writes the workgroup's partial
//                   dW1 = X^T dZ1, dW2 = H^T dZ2 and sum of squared residuals
//                   to its slot.
//   k_reduce<H>     sums the slots in slot order (deterministic), then either
//                   writes dW1/dW2/loss or applies W -= lr dW (eq. 19) and
//                   records the step and epoch loss.
// The persistent single-launch trainer lives in train_persistent.hip, the
// forward pass of mlp_forward in forward.hip.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

// ---------------------------------------------------------------------------
// Tile kernels
// ---------------------------------------------------------------------------

constexpr int RG = 8;  // rows staged per LDS round

template <int H>
struct TileShape {
    static constexpr int NT = H < 64 ? 64 : H;  // threads per workgroup
    static constexpr int NW = NT / 64;          // waves per workgroup
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// Row index of batch position t: idx[off + t] or off + t. Out-of-range rows are
// replaced by row 0 and flagged.
__device__ __forceinline__ int64_t fetch_row(const int32_t *__restrict__ idx, int64_t off,
                                             int64_t t, int64_t n_rows, int32_t *err) {
    int64_t r = idx ? (int64_t)idx[off + t] : off + t;
    if (r < 0 || r >= n_rows) {
        __hip_atomic_store(err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r = 0;
    }
    return r;
}

template <int H>
__global__ __launch_bounds__(TileShape<H>::NT) void k_tile(
    const float *__restrict__ X, int64_t n_rows, const float *__restrict__ Y,
    const int32_t *__restrict__ idx, int64_t idx_off, int64_t nb, int rows_per_wg,
    const float *__restrict__ W1, const float *__restrict__ W2, float *__restrict__ partial,
    int64_t slot_stride, int32_t *err) {
    constexpr int NT = TileShape<H>::NT;
    constexpr int NW = TileShape<H>::NW;
    __shared__ float xs[RG][D_IN];
    __shared__ float ys[RG];
    __shared__ float red[RG][NW];
    __shared__ float yp[RG];

    const int j = threadIdx.x;
    const int lane = j & 63, wave = j >> 6;
    const bool unit = j < H;
    float w1[D_IN], p[D_IN];
#pragma unroll
    for (int k = 0; k < D_IN; ++k) {
        w1[k] = unit ? W1[k * H + j] : 0.0f;
        p[k] = 0.0f;
    }
    const float w2 = unit ? W2[j] : 0.0f;
    float q = 0.0f, sse = 0.0f;
    const float scale = 2.0f / (float)nb;

    const int64_t t0 = (int64_t)blockIdx.x * rows_per_wg;
    const int64_t t1 = t0 + rows_per_wg < nb ? t0 + rows_per_wg : nb;
    for (int64_t tg = t0; tg < t1; tg += RG) {
        // Stage RG rows (zero rows past the end contribute nothing: z = 0, y = 0).
        for (int e = j; e < RG * D_IN; e += NT) {
            const int rr = e / D_IN, k = e % D_IN;
            const int64_t t = tg + rr;
            float v = 0.0f;
            if (t < t1) v = X[fetch_row(idx, idx_off, t, n_rows, err) * D_IN + k];
            xs[rr][k] = v;
        }
        if (j < RG) {
            const int64_t t = tg + j;
            float v = 0.0f;
            if (t < t1) v = Y[fetch_row(idx, idx_off, t, n_rows, err)];
            ys[j] = v;
        }
        __syncthreads();

        float z[RG];
#pragma unroll
        for (int rr = 0; rr < RG; ++rr) {
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < D_IN; ++k) acc = fmaf(xs[rr][k], w1[k], acc);   // eq. 11
            z[rr] = acc;
            const float a = wave_sum((acc > 0.0f ? acc : 0.0f) * w2);           // eqs. 12-13
            if (lane == 0) red[rr][wave] = a;
        }
        __syncthreads();
        if (j < RG) {
            float s = 0.0f;
#pragma unroll
            for (int w = 0; w < NW; ++w) s += red[j][w];
            yp[j] = s;
        }
        __syncthreads();
#pragma unroll
        for (int rr = 0; rr < RG; ++rr) {
            const float res = yp[rr] - ys[rr];
            const float g = scale * res;                                        // eq. 15
            if (j == 0) sse = fmaf(res, res, sse);                              // eq. 14
            const bool on = z[rr] > 0.0f;                                       // ReLU'(z) = [z > 0]
            q = fmaf(on ? z[rr] : 0.0f, g, q);                                  // eq. 16
            const float dz = on ? g * w2 : 0.0f;                                // eq. 17
#pragma unroll
            for (int k = 0; k < D_IN; ++k) p[k] = fmaf(xs[rr][k], dz, p[k]);     // eq. 18
        }
        __syncthreads();
    }
    float *slot = partial + (int64_t)blockIdx.x * slot_stride;
    if (unit) {
#pragma unroll
        for (int k = 0; k < D_IN; ++k) slot[k * H + j] = p[k];
        slot[D_IN * H + j] = q;
    }
    if (j == 0) slot[(D_IN + 1) * H] = sse;
}

// Fixed-order reduction of G slots. Thread t owns output t of the flattened
// [dW1 (d*H) | dW2 (H) | sse (1)] vector.
template <int H>
__global__ __launch_bounds__(256) void k_reduce(const float *__restrict__ partial, int G,
                                                int64_t slot_stride, ReduceArgs a) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    constexpr int N1 = D_IN * H;
    if (t > N1 + H) return;
    float s = 0.0f;
    for (int g = 0; g < G; ++g) s += partial[(int64_t)g * slot_stride + t];
    if (t < N1) {
        if (a.sgd) a.W1[t] -= a.lr * s;                                         // eq. 19
        else a.dW1[t] = s;
    } else if (t < N1 + H) {
        if (a.sgd) a.W2[t - N1] -= a.lr * s;
        else a.dW2[t - N1] = s;
    } else {
        const float L = s * a.inv_nb;                                            // eq. 14
        flag_nonfinite(s, &a.ctl->err);
        if (a.loss) a.loss[0] = L;
        if (a.step_loss) a.step_loss[a.step] = L;
        if (a.epoch_loss) {
            double acc = a.first_in_epoch ? 0.0 : a.ctl->epoch_sse;
            acc += (double)s;
            a.ctl->epoch_sse = acc;
            a.epoch_loss[a.epoch] = (float)(acc * a.inv_n);
        }
    }
}

__global__ void k_fill(float *p, int64_t n, float v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_clear_ctl(Control *c) {
    if (blockIdx.x == 0) {
        if (threadIdx.x == 0) {
            c->err = 0;
            c->abort = 0;
            c->epoch_sse = 0.0;
        }
        c->reg[threadIdx.x] = 0;   // 64 threads
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers for the tile path
// ---------------------------------------------------------------------------

template <int H>
static hipError_t launch_tile(const Ctx &c, const float *X, int64_t n_rows, const float *Y,
                              const int32_t *idx, int64_t idx_off, int64_t nb, int rows_per_wg,
                              int G) {
    constexpr int NT = TileShape<H>::NT;
    hipLaunchKernelGGL((k_tile<H>), dim3(G), dim3(NT), 0, c.stream, X, n_rows, Y, idx, idx_off, nb,
                       rows_per_wg, c.W1, c.W2, c.slots, c.slot_stride, &c.ctl->err);
    return hipGetLastError();
}

template <int H>
static hipError_t launch_reduce(const Ctx &c, int G, const ReduceArgs &a) {
    const int n = D_IN * H + H + 1;
    hipLaunchKernelGGL((k_reduce<H>), dim3((n + 255) / 256), dim3(256), 0, c.stream, c.slots, G,
                       c.slot_stride, a);
    return hipGetLastError();
}

#define MLP_DISPATCH_H(h, CALL)                 \
    switch (h) {                                \
    case 32: { constexpr int HH = 32; CALL; }   \
    case 64: { constexpr int HH = 64; CALL; }   \
    case 128: { constexpr int HH = 128; CALL; } \
    case 256: { constexpr int HH = 256; CALL; } \
    case 512: { constexpr int HH = 512; CALL; } \
    case 1024: { constexpr int HH = 1024; CALL; } \
    default: return hipErrorInvalidValue;       \
    }

// Rows per workgroup for a batch of nb rows: at most TILE_SLOTS workgroups.
int tile_rows_per_wg(int64_t nb) {
    int64_t r = (nb + TILE_SLOTS - 1) / TILE_SLOTS;
    r = (r + RG - 1) / RG * RG;
    return (int)(r < RG ? RG : r);
}

hipError_t tile_step(const Ctx &c, const float *X, int64_t n_rows, const float *Y,
                     const int32_t *idx, int64_t idx_off, int64_t nb, const ReduceArgs &a) {
    const int R = tile_rows_per_wg(nb);
    const int G = (int)((nb + R - 1) / R);
    hipError_t e;
    MLP_DISPATCH_H(c.hidden, {
        e = launch_tile<HH>(c, X, n_rows, Y, idx, idx_off, nb, R, G);
        if (e != hipSuccess) return e;
        return launch_reduce<HH>(c, G, a);
    });
}

hipError_t clear_control(const Ctx &c) {
    hipLaunchKernelGGL(k_clear_ctl, dim3(1), dim3(64), 0, c.stream, c.ctl);
    return hipGetLastError();
}

__global__ void k_zero64(uint64_t *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

hipError_t clear_words(const Ctx &c, uint64_t *p, int64_t n) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_zero64, dim3(1024), dim3(256), 0, c.stream, p, n);
    return hipGetLastError();
}

hipError_t fill(const Ctx &c, float *p, int64_t n, float v) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, c.stream, p, n, v);
    return hipGetLastError();
}

}  // namespace mlp
