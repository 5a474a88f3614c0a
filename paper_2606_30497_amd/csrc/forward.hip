// forward.hip -- the forward pass over many rows (eqs. 11-13), for inference
// and full-dataset evaluation (mlp_forward), with fp32 products formed on the
// bf16 matrix cores.
//
// Per sample the pass is 2 * 32 * h FLOP of the layer-1 contraction plus 2 h
// of the output product against 132 bytes of HBM traffic (an X row and its
// output; 4 more with a row index).
//
// The 32-deep contraction of a 16-row tile with a 16-unit tile is one
// v_mfma_f32_16x16x32_bf16 per part product: X and W1 are split into three
// bf16 parts each (bf16x3.h) and the six part products with i + j <= 2 are
// accumulated in fp32, smallest first -- six 16-cycle MFMAs where fp32 MFMA
// takes eight of 32 cycles, and a bf16 MFMA does not hold up the other waves
// of its SIMD.
//
// A wave keeps the split weights of up to 128 hidden units in registers for its
// whole life (three parts of W1[8 lq .. 8 lq + 7][unit] per unit tile, 12
// VGPRs, plus one W2 value) and streams 16-row tiles of X:
//   lane (li, lq) = (lane % 16, lane / 16) loads X[row li][8 lq .. 8 lq + 7]
//   (two 16-byte loads), which is its A operand of the MFMA, and splits it; the
//   MFMAs accumulate Z1[4 lq + v][unit 16 u + li] of unit tile u in acc[u][v];
//   ReLU and the W2 product stay in registers (eqs. 12-13), and a DPP
//   butterfly sums each row's 16 unit lanes.
// For h > 128 the waves of a workgroup split the units of one row tile and add
// their partial outputs in LDS in a fixed order. The next tile's rows are
// loaded while the current tile is on the matrix cores.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "bf16x3.h"
#include "lanes.h"
#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

template <int H>
struct FwdShape {
    static constexpr int UW = H < 128 ? H : 128;   // units per wave
    static constexpr int NUT = UW / 16;            // unit tiles per wave
    static constexpr int WPT = H / UW;             // waves per row tile: 1, 2, 4 or 8
    static constexpr int WAVES = WPT > 4 ? WPT : 4;   // waves per workgroup
    static constexpr int TPI = WAVES / WPT;        // row-tile slots per workgroup iteration
    // row tiles per slot and iteration: the HBM-bound h = 32 keeps four tiles
    // of loads in flight per wave (at four waves a SIMD)
    static constexpr int RT = H == 32 ? 4 : 1;
    // waves per SIMD the register budget allows (a wave holds 13 registers per
    // unit tile of weights and 4 of accumulators, about 40 more, and 8 per row
    // tile in flight): small nets need enough row loads outstanding; at
    // 128 units a wave, three (168 registers, a few of them spilled) beat two
    // (172) where a workgroup's waves fit three times, i.e. except at h = 1024
    // (eight waves a workgroup)
    static constexpr int WAVES_PER_SIMD = NUT <= 4 ? 4 : WPT == 8 ? 2 : 3;
    static_assert(H % 16 == 0 && WPT * UW == H && WPT <= 8, "shape");
};

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
__global__ __launch_bounds__(64 * FwdShape<H>::WAVES, FwdShape<H>::WAVES_PER_SIMD) void k_forward(
    const float *__restrict__ X, int64_t n_rows, const int32_t *__restrict__ idx, int64_t B,
    const float *__restrict__ W1, const float *__restrict__ W2, float *__restrict__ ypred,
    int32_t *err) {
    using S = FwdShape<H>;
    constexpr int NUT = S::NUT, WPT = S::WPT, TPI = S::TPI, RT = S::RT;
    __shared__ float part[S::WAVES][16];   // partial outputs of the waves of a row tile (WPT > 1)

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15, lq = lane >> 4;
    const int wt = wave / WPT;   // row-tile slot within an iteration
    const int wu = wave % WPT;   // unit block: units [wu * UW, wu * UW + UW)

    // the wave's weights, for its whole life: the parts of W1[8 lq + t][unit]
    // (t = 0..7), and W2[unit]
    u4v w1p[NUT][3];
    float w2v[NUT];
#pragma unroll
    for (int u = 0; u < NUT; ++u) {
        const int unit = wu * S::UW + 16 * u + li;
        uint32_t w[4][3];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            split_pair(W1[(8 * lq + 2 * t) * H + unit], W1[(8 * lq + 2 * t + 1) * H + unit], w[t]);
#pragma unroll
        for (int p = 0; p < 3; ++p) w1p[u][p] = u4v{w[0][p], w[1][p], w[2][p], w[3][p]};
        w2v[u] = W2[unit];
    }

    // one 16-row tile rt at batch row r0: eq. 11 (the six part products
    // smallest first, every unit tile's product of one part pair back to back),
    // ReLU and the W2 product in registers (eqs. 12-13), the row sums out
    auto tile = [&](const RowTile &rt, int64_t r0) __attribute__((always_inline)) {
        u4v xp[3];
        {
            uint32_t w[4][3];
#pragma unroll
            for (int t = 0; t < 4; ++t) split_pair(rt.x[2 * t], rt.x[2 * t + 1], w[t]);
#pragma unroll
            for (int p = 0; p < 3; ++p) xp[p] = u4v{w[0][p], w[1][p], w[2][p], w[3][p]};
        }
        constexpr int PA[6] = {2, 1, 0, 1, 0, 0}, PB[6] = {0, 1, 2, 0, 1, 0};
        f4 acc[NUT];
#pragma unroll
        for (int u = 0; u < NUT; ++u) acc[u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < 6; ++q)
#pragma unroll
            for (int u = 0; u < NUT; ++u) acc[u] = mfma_bf16(xp[PA[q]], w1p[u][PB[q]], acc[u]);
        // the lane's share of Ypred for rows 4 lq + v, units ascending
        float yp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < NUT; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                // ReLU as an integer max on the bits: every negative float
                // (-0 included) has a negative pattern and becomes +0, every
                // positive one stays; one instruction, where the float form
                // costs two (a canonicalizing max first)
                const float z = __int_as_float(max(__float_as_int(acc[u][v]), 0));
                yp[v] = fmaf(z, w2v[u], yp[v]);
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
    };

    // iteration it: tiles (it TPI + wt) RT + j, j < RT, of this wave
    const int64_t ntiles = (B + 15) / 16;
    const int64_t iters = (ntiles + TPI * RT - 1) / (TPI * RT);
    auto row0 = [&](int64_t i, int j) { return ((i * TPI + wt) * RT + j) * 16; };
    int64_t it = blockIdx.x;
    RowTile cur[RT];
    int32_t ixn[RT];
#pragma unroll
    for (int j = 0; j < RT; ++j) {
        cur[j] = load_rows(X, n_rows, idx, B, row0(it, j), load_index(idx, B, row0(it, j) + li), li, lq, err);
        ixn[j] = load_index(idx, B, row0(it + gridDim.x, j) + li);
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    for (; it < iters; it += gridDim.x) {
        // the next iteration's rows, in flight while these tiles are computed,
        // and the indices of the iteration after it
        RowTile nxt[RT];
#pragma unroll
        for (int j = 0; j < RT; ++j) {
            nxt[j] = load_rows(X, n_rows, idx, B, row0(it + gridDim.x, j), ixn[j], li, lq, err);
            ixn[j] = load_index(idx, B, row0(it + 2 * (int64_t)gridDim.x, j) + li);
        }
#pragma unroll
        for (int j = 0; j < RT; ++j) tile(cur[j], row0(it, j));
#pragma unroll
        for (int j = 0; j < RT; ++j) cur[j] = nxt[j];
    }
}

template <int H>
static hipError_t launch_forward_h(const Ctx &c, const float *X, int64_t n_rows,
                                   const int32_t *idx, int64_t B, float *ypred) {
    using S = FwdShape<H>;
    const int64_t ntiles = (B + 15) / 16;
    const int64_t iters = (ntiles + S::TPI * S::RT - 1) / (S::TPI * S::RT);
    // resident workgroups: WAVES_PER_SIMD waves on each of a CU's four SIMDs
    const int64_t cap = (int64_t)S::WAVES_PER_SIMD * 4 / S::WAVES * (c.num_cu > 0 ? c.num_cu : 256);
    const int grid = (int)(iters < cap ? iters : cap);
    hipLaunchKernelGGL((k_forward<H>), dim3(grid), dim3(64 * S::WAVES), 0, c.stream, X, n_rows, idx,
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
