// forward.hip -- the forward pass over many rows (eqs. 11-13) on fp32 MFMA,
// for inference and full-dataset evaluation (mlp_forward).
//
// Per sample the pass is 2 * 32 * h FLOP of the layer-1 contraction plus 2 h
// of the output product against 132 bytes of HBM traffic (an X row and its
// output; 4 more with a row index): at ~128 FLOP/byte for h = 256 it is a dense
// contraction bound by the matrix cores, not by HBM.
//
// A wave keeps the weights of up to 256 hidden units in registers for its whole
// life, as the B operands of v_mfma_f32_16x16x4f32 (16 unit tiles x 8 k steps)
// plus one W2 value per unit tile, and streams 16-row tiles of X:
//   lane (li, lq) = (lane % 16, lane / 16) loads X[row li][8 lq .. 8 lq + 7]
//   (two 16-byte loads) and feeds k = 8 lq + t to MFMA step t, so eight MFMAs
//   accumulate Z1[4 lq + v][unit 16 u + li] of unit tile u in acc[u][v];
//   ReLU and the W2 product stay in registers (eqs. 12-13), and a DPP
//   butterfly sums each row's 16 unit lanes.
// For h > 256 the waves of a workgroup split the units of one row tile and add
// their partial outputs in LDS in a fixed order. The next tile's rows are
// loaded while the current tile is on the matrix cores.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "lanes.h"
#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

template <int H>
struct FwdShape {
    static constexpr int UW = H < 256 ? H : 256;   // units per wave
    static constexpr int NUT = UW / 16;            // unit tiles per wave
    static constexpr int WPT = H / UW;             // waves per row tile: 1, 2 or 4
    static constexpr int TPI = 4 / WPT;            // row tiles per workgroup iteration
    // workgroups per CU the register budget allows (a wave holds 8.5 UW weight
    // registers plus 4 NUT accumulators): small nets need more waves in flight
    // to keep enough row loads outstanding
    static constexpr int WG_PER_CU = UW <= 32 ? 8 : UW <= 64 ? 4 : UW <= 128 ? 3 : 2;
    static_assert(H % 16 == 0 && WPT * UW == H && (WPT == 1 || WPT == 2 || WPT == 4), "shape");
};

constexpr int FWD_THREADS = 256;

// Rows of one 16-row tile as MFMA A operands: lane (li, lq) holds
// X[r_t][8 lq .. 8 lq + 7] of batch position t = r0 + li (zeros past B).
struct RowTile {
    float x[8];
};

// The batch index of tile row t, loaded ahead of the rows it selects (an
// unconditional load from a clamped address; only read for t < B).
__device__ __forceinline__ int32_t load_index(const int32_t *__restrict__ idx, int64_t B, int64_t t) {
    return idx ? idx[t < B ? t : B - 1] : 0;
}
// Rows r0 + li (t < B) of X, through the index ix loaded for them.
__device__ __forceinline__ RowTile load_rows(const float *__restrict__ X, int64_t n_rows,
                                             const int32_t *__restrict__ idx, int64_t B, int64_t r0,
                                             int32_t ix, int li, int lq, int32_t *err) {
    RowTile rt;
    const int64_t t = r0 + li;
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
    if (t < B) {
        int64_t r = idx ? (int64_t)ix : t;
        if (r < 0 || r >= n_rows) {
            __hip_atomic_store(err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            r = 0;
        }
        const float4 *p = reinterpret_cast<const float4 *>(X + r * D_IN + 8 * lq);
        a = p[0];
        b = p[1];
    }
    rt.x[0] = a.x; rt.x[1] = a.y; rt.x[2] = a.z; rt.x[3] = a.w;
    rt.x[4] = b.x; rt.x[5] = b.y; rt.x[6] = b.z; rt.x[7] = b.w;
    return rt;
}

template <int H>
__global__ __launch_bounds__(FWD_THREADS, FwdShape<H>::WG_PER_CU) void k_forward(
    const float *__restrict__ X, int64_t n_rows, const int32_t *__restrict__ idx, int64_t B,
    const float *__restrict__ W1, const float *__restrict__ W2, float *__restrict__ ypred,
    int32_t *err) {
    using S = FwdShape<H>;
    constexpr int NUT = S::NUT, WPT = S::WPT, TPI = S::TPI;
    __shared__ float part[4][16];   // partial outputs of the waves of a row tile (WPT > 1)

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15, lq = lane >> 4;
    const int wt = wave / WPT;   // row-tile slot within an iteration
    const int wu = wave % WPT;   // unit block: units [wu * 256, wu * 256 + 256)

    // the wave's weights, for its whole life: W1[8 lq + t][unit], W2[unit]
    float w1b[NUT][8], w2v[NUT];
#pragma unroll
    for (int u = 0; u < NUT; ++u) {
        const int unit = wu * S::UW + 16 * u + li;
#pragma unroll
        for (int t = 0; t < 8; ++t) w1b[u][t] = W1[(8 * lq + t) * H + unit];
        w2v[u] = W2[unit];
    }

    const int64_t ntiles = (B + 15) / 16;
    const int64_t iters = (ntiles + TPI - 1) / TPI;
    int64_t it = blockIdx.x;
    const int64_t r0f = (it * TPI + wt) * 16;
    RowTile cur = load_rows(X, n_rows, idx, B, r0f, load_index(idx, B, r0f + li), li, lq, err);
    int32_t ixn = load_index(idx, B, ((it + gridDim.x) * TPI + wt) * 16 + li);
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    for (; it < iters; it += gridDim.x) {
        const int64_t r0 = (it * TPI + wt) * 16;
        // the next iteration's rows, in flight while this tile is computed, and
        // the index of the iteration after it
        const int64_t r0n = ((it + gridDim.x) * TPI + wt) * 16;
        const RowTile nxt = load_rows(X, n_rows, idx, B, r0n, ixn, li, lq, err);
        ixn = load_index(idx, B, ((it + 2 * (int64_t)gridDim.x) * TPI + wt) * 16 + li);

        // eq. 11: Z1 tile = X tile W1 (8 k steps of 4 per unit tile)
        f4 acc[NUT];
#pragma unroll
        for (int u = 0; u < NUT; ++u) acc[u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
            for (int u = 0; u < NUT; ++u)
                acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur.x[t], w1b[u][t], acc[u], 0, 0, 0);
        // eqs. 12-13: the lane's share of Ypred for rows 4 lq + v, units ascending
        float yp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < NUT; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float z = acc[u][v];
                yp[v] = fmaf(z > 0.0f ? z : 0.0f, w2v[u], yp[v]);
            }
        // lane li ends with row 4 lq + (li >> 2) summed over the 16 unit lanes
        const float rowv = rsum16x4(yp, li);
        const int rr = 4 * lq + (li >> 2);
        if constexpr (WPT == 1) {
            if ((li & 3) == 0 && r0 + rr < B) ypred[r0 + rr] = rowv;
        } else {
            if ((li & 3) == 0) part[wave][rr] = rowv;
            __syncthreads();
            if (wu == 0 && lane < 16 && r0 + lane < B) {
                float s = 0.0f;
#pragma unroll
                for (int w = 0; w < WPT; ++w) s += part[wt * WPT + w][lane];
                ypred[r0 + lane] = s;
            }
            __syncthreads();
        }
        cur = nxt;
    }
}

template <int H>
static hipError_t launch_forward_h(const Ctx &c, const float *X, int64_t n_rows,
                                   const int32_t *idx, int64_t B, float *ypred) {
    using S = FwdShape<H>;
    const int64_t ntiles = (B + 15) / 16;
    const int64_t iters = (ntiles + S::TPI - 1) / S::TPI;
    const int64_t cap = S::WG_PER_CU * (int64_t)(c.num_cu > 0 ? c.num_cu : 256);
    const int grid = (int)(iters < cap ? iters : cap);
    hipLaunchKernelGGL((k_forward<H>), dim3(grid), dim3(FWD_THREADS), 0, c.stream, X, n_rows, idx,
                       B, c.W1, c.W2, ypred, &c.ctl->err);
    return hipGetLastError();
}

hipError_t launch_forward(const Ctx &c, const float *X, int64_t n_rows, const int32_t *idx,
                          int64_t B, float *ypred) {
    switch (c.hidden) {
    case 32: return launch_forward_h<32>(c, X, n_rows, idx, B, ypred);
    case 64: return launch_forward_h<64>(c, X, n_rows, idx, B, ypred);
    case 128: return launch_forward_h<128>(c, X, n_rows, idx, B, ypred);
    case 256: return launch_forward_h<256>(c, X, n_rows, idx, B, ypred);
    case 512: return launch_forward_h<512>(c, X, n_rows, idx, B, ypred);
    case 1024: return launch_forward_h<1024>(c, X, n_rows, idx, B, ypred);
    }
    return hipErrorInvalidValue;
}

}  // namespace mlp
