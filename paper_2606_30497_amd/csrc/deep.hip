// deep.hip -- mini-batch SGD for a 32-h-...-h-1 ReLU/MSE network with L hidden
// layers (the deeper networks the paper leaves to future work, Sec. VII.B), on
// gfx950. The step is the paper's eqs. 11-19 applied layer by layer with the
// layer index of eq. 9:
//   H_0 = X_b;  H_l = ReLU(H_{l-1} W_l), l = 1..L;  Ypred = H_L w_o
//   dZ_o = (2/n_b)(Ypred - Y);  dw_o = H_L^T dZ_o;  G_L = (dZ_o w_o^T) (.) [H_L > 0]
//   dW_l = H_{l-1}^T G_l;  G_{l-1} = (G_l W_l^T) (.) [H_{l-1} > 0]   (l >= 2)
//   every parameter -= lr * its gradient, after all gradients are formed.
// ([H > 0] equals [Z > 0] since H = max(Z, 0), so the pre-activations are never
// stored.)
//
// Unlike the one-layer trainer, the hidden-to-hidden products are real GEMMs
// ([n_b x h] x [h x h], 2 n_b h^2 FLOP each), so the step is a sequence of
// MFMA GEMM launches from the host, with the activations of the batch in the
// workspace:
//   k_gemm<NN, RELU>   the forward of a layer, ReLU in the epilogue
//   k_gemm<TN, NONE>   dW_l = H_{l-1}^T G_l, split over row chunks (grid z);
//                      each chunk writes its own partial, summed in chunk order
//   k_gemm<NT, MASK>   G_{l-1} = (G_l W_l^T) masked by H_{l-1} > 0; into
//                      layer 1 its epilogue also forms each row tile's
//                      partial of dW_1 = X^T G_1 (no launch of its own)
//   k_gemm_pair        the weight gradient and the back-propagation of one
//                      layer (both read G_l, neither reads the other's output)
//                      in one launch
//   k_deep_out         Ypred, residual, dZ_o, G_L and the dw_o partial of a
//                      chunk of rows (one wave per row)
//   k_deep_apply       sums every gradient's chunk partials in order and
//                      applies eq. 19 (or writes the gradients); one workgroup
//                      reduces the batch loss in a fixed tree, and in a training
//                      loop the last ones gather the next step's rows
// Every output element is one lane's sum in a fixed order, so results are
// bitwise reproducible.
//
// GEMM tile: 64 x 64 (or 32 x 64, 32 x 32) outputs per workgroup of four waves
// (each a quarter, as 16 x 16 MFMA tiles), K in chunks of 32 staged in LDS,
// alternating between two LDS buffers (one barrier per chunk); the next two
// chunks' global loads are in flight while the current chunk is computed. Two
// flavours of the product:
// - fp32: v_mfma_f32_16x16x4f32 on fp32 operands (in LDS, operands read along
//   m or n stored k-major with a row stride of TM + 16 floats, operands read
//   along k as loaded with a stride of 34, so that MFMA operand reads are
//   conflict-free);
// - bf16x3: fp32 products formed on the bf16 matrix cores. Each operand is
//   split once, as it is staged, into three bf16 parts (x = x0 + x1 + x2
//   exactly, each part the rounding to nearest of what the earlier parts
//   leave), and a b is the sum of the six part products a_i b_j with
//   i + j <= 2, each exact in fp32, accumulated by v_mfma_f32_16x16x32_bf16 in
//   fp32: a0 b0 in one sum, the other five in a second, added at the end. The
//   dropped part products are below 2.01 u |a b| (u = 2^-24); the second sum's
//   terms are below 2^-7 |a b| together, so its roundings add about 0.04 K u to
//   the K u of an fp32 dot product of length K. Six bf16 MFMAs of 16 cycles
//   replace eight fp32 MFMAs of 32 cycles per 32-deep chunk of a 16 x 16 tile,
//   and a bf16 MFMA does not hold up the other waves of its SIMD while it runs,
//   as an fp32 one does; the split costs VALU work and LDS space (the parts as
//   [3][T][32] bf16, k inner, 16-byte granules permuted by row so that operand
//   reads and staging writes are conflict-free).
#include <hip/hip_runtime.h>

#include <math.h>
#include <new>
#include <stdint.h>
#include <string.h>

#include "bf16x3.h"
#include "lanes.h"
#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

constexpr int GT = 64;        // GEMM tile (M and N)
constexpr int GK = 32;        // K chunk
constexpr int GMS = 34;       // LDS row stride of an x-major fp32 operand tile ([x][k], floats)
constexpr int GSTAGES = 2;    // K chunks in flight (register stages; 3 or 4 measured slower)
constexpr int GEMM_CUS = 256; // compute units the tile choice plans for
constexpr int SPLIT_MAX = 64; // row chunks of a weight-gradient product
constexpr int OUT_CHUNKS_MAX = 256;   // row chunks of the output layer (dw_o partials)
constexpr int DEEP_MAX_LAYERS = 8;

enum { OP_NN = 0, OP_TN = 1, OP_NT = 2 };
// Epilogues: none; ReLU (eq. 12); the ReLU mask of eq. 17; the mask and, from
// the masked tile, the tile's share of dW_1 = X^T G_1 (eq. 18 for the first
// layer, see gemm_block)
enum { EP_NONE = 0, EP_RELU = 1, EP_MASK = 2, EP_MASK_DW1 = 3 };

// Global -> register staging of one K chunk of a TM x TN output tile: each of
// the 256 threads holds TM / 8 values of the a tile ([TM x 32]) and TN / 8 of
// the b tile ([32 x TN]).
template <int TM, int TN>
struct Stage {
    float4 a[TM / 32], b[TN / 32];
};

// Sixteen zero bytes in device memory: a lane whose value lies outside its
// operand loads these instead. The choice is made on the address, before the
// load, and the loaded registers are not touched again until they are written
// to LDS. (A load under a lane condition compiles to a branch and an immediate
// wait for that load; a select of zero after the load is consumed, and so
// waited for, wherever the scheduler places it, often among the MFMAs of an
// earlier chunk. Either way the next chunks' loads stop overlapping the current
// chunk's MFMAs.)
__device__ __attribute__((aligned(16))) float g_zero16[4] = {0.f, 0.f, 0.f, 0.f};

__device__ __forceinline__ float4 ld4(bool ok, const float *p) {
    return *reinterpret_cast<const float4 *>(ok ? p : g_zero16);
}
__device__ __forceinline__ float ld1(bool ok, const float *p) { return *(ok ? p : g_zero16); }

// ---- fp32 flavour: operands staged as fp32, v_mfma_f32_16x16x4f32 ----------
//
// LDS row stride of a k-major operand tile of width T ([k][x], floats): T + 16,
// so that the four k rows an MFMA operand read touches per wave fall in four
// different groups of 16 banks.
__host__ __device__ constexpr int kmajor_stride(int T) { return T + 16; }
// floats of one fp32 LDS operand tile of width T (k-major [32][T + 16] or
// x-major [T][GMS])
__host__ __device__ constexpr int f32_tile_floats(int T) {
    return GK * kmajor_stride(T) > T * GMS ? GK * kmajor_stride(T) : T * GMS;
}

// One operand tile of width T (T = 32 or 64; x is m for the a tile, n for the
// b tile) and K chunk [k0, k0 + 32), thread t's float4 h (h < T / 32):
//   loaded along x (k-major operand, P[k ld + x]):
//     (k, x) = (t / (T/4) + (1024/T) h, 4 (t % (T/4)))
//   loaded along k (x-major operand, P[x ld + k]):
//     (x, k) = (t / (256/T), 4 (t % (256/T)) + (1024/T) h)
template <bool KMAJOR, int T>
__device__ __forceinline__ void fetch_f32(float4 (&r)[T / 32], const float *__restrict__ P, int ld,
                                          int64_t xlim, int64_t x0, int64_t k0, int64_t ke, int t) {
#pragma unroll
    for (int h = 0; h < T / 32; ++h) {
        if constexpr (KMAJOR) {
            const int64_t k = k0 + t / (T / 4) + (1024 / T) * h, x = x0 + (t % (T / 4)) * 4;
            r[h] = ld4(k < ke && x < xlim, P + k * ld + x);
        } else {
            const int64_t x = x0 + t / (256 / T), k = k0 + (t % (256 / T)) * 4 + (1024 / T) * h;
            r[h] = ld4(x < xlim && k < ke, P + x * ld + k);
        }
    }
}

// Registers -> LDS: a k-major operand is stored as loaded, [k][x] with stride
// T + 16; an x-major one as loaded too, [x][k] with stride GMS = 34 (the 16 x
// rows x 2 k columns an MFMA operand read touches per half wave land in 32
// distinct banks), in 8-byte stores (the stride is not a multiple of 4).
template <bool KMAJOR, int T>
__device__ __forceinline__ void stash_f32(const float4 (&r)[T / 32], float *S, int t) {
#pragma unroll
    for (int h = 0; h < T / 32; ++h) {
        if constexpr (KMAJOR) {
            *reinterpret_cast<float4 *>(S + (t / (T / 4) + (1024 / T) * h) * kmajor_stride(T) +
                                        (t % (T / 4)) * 4) = r[h];
        } else {
            float2 *d = reinterpret_cast<float2 *>(S + (t / (256 / T)) * GMS + (t % (256 / T)) * 4 +
                                                   (1024 / T) * h);
            d[0] = make_float2(r[h].x, r[h].y);
            d[1] = make_float2(r[h].z, r[h].w);
        }
    }
}

// ---- bf16x3 flavour: operands split into three bf16 parts, bf16 MFMA --------
//
// floats (4-byte words) of one split LDS operand tile of width T: three bf16
// parts of [T][32], k inner
__host__ __device__ constexpr int bf3_tile_floats(int T) { return 3 * T * GK / 2; }

// Position in its row of element k of row x: the row's four 16-byte granules
// are permuted by (x >> 2) & 3, so that 8 consecutive rows read at one granule,
// and 16 rows written at one 8-byte half granule, fall in distinct banks.
__device__ __forceinline__ int swz(int x, int k) { return (((k >> 3) ^ ((x >> 2) & 3)) << 3) | (k & 7); }

// Thread t holds E = T / 8 values of one row x and k in [kr, kr + E):
//   loaded along x (k-major operand, P[k ld + x]; a wave's lanes take
//   consecutive x, so each of the E scalar loads is one contiguous row segment):
//     x = t % T, kr = E (t / T)
//   loaded along k (x-major operand, P[x ld + k]; E / 4 float4 loads):
//     x = t / (32 / E), kr = E (t % (32 / E))
template <bool KMAJOR, int T>
__device__ __forceinline__ void fetch_bf3(float4 (&r)[T / 32], const float *__restrict__ P, int ld,
                                          int64_t xlim, int64_t x0, int64_t k0, int64_t ke, int t) {
    static_assert(T == 32 || T == 64, "operand tile width");
    constexpr int E = T / 8;
    if constexpr (KMAJOR) {
        const int64_t x = x0 + t % T, k = k0 + E * (t / T);
        float v[E];
#pragma unroll
        for (int j = 0; j < E; ++j) v[j] = ld1(x < xlim && k + j < ke, P + (k + j) * ld + x);
#pragma unroll
        for (int h = 0; h < T / 32; ++h) r[h] = make_float4(v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]);
    } else {
        const int64_t x = x0 + t / (32 / E), k = k0 + E * (t % (32 / E));
#pragma unroll
        for (int h = 0; h < T / 32; ++h) r[h] = ld4(x < xlim && k + 4 * h < ke, P + x * ld + k + 4 * h);
    }
}

// Registers -> LDS: the thread's E values split into three bf16 parts, part p
// written to row x of part tile p at swz(x, kr) in one 16-byte (E = 8) or
// 8-byte (E = 4) store.
template <bool KMAJOR, int T>
__device__ __forceinline__ void stash_bf3(const float4 (&r)[T / 32], uint16_t *S, int t) {
    constexpr int E = T / 8;
    const int x = KMAJOR ? t % T : t / (32 / E), kr = KMAJOR ? E * (t / T) : E * (t % (32 / E));
    uint32_t w[3][E / 2];
#pragma unroll
    for (int h = 0; h < T / 32; ++h) {
        uint32_t q[3];
        split_pair(r[h].x, r[h].y, q);
#pragma unroll
        for (int p = 0; p < 3; ++p) w[p][2 * h] = q[p];
        split_pair(r[h].z, r[h].w, q);
#pragma unroll
        for (int p = 0; p < 3; ++p) w[p][2 * h + 1] = q[p];
    }
#pragma unroll
    for (int p = 0; p < 3; ++p) {
        uint16_t *d = S + (p * T + x) * GK + swz(x, kr);
        if constexpr (E == 8)
            *reinterpret_cast<u4v *>(d) = u4v{w[p][0], w[p][1], w[p][2], w[p][3]};
        else
            *reinterpret_cast<u2v *>(d) = u2v{w[p][0], w[p][1]};
    }
}

// ---- the product ---------------------------------------------------------------

// floats of one LDS operand tile of width T in either flavour
__host__ __device__ constexpr int tile_floats(int T, bool bf3) {
    return bf3 ? bf3_tile_floats(T) : f32_tile_floats(T);
}

template <int OP, int TM, int TN, bool BF3>
__device__ __forceinline__ void gemm_fetch(Stage<TM, TN> &st, const float *__restrict__ A, int lda,
                                           const float *__restrict__ B, int ldb, int64_t M, int N,
                                           int64_t m0, int n0, int64_t k0, int64_t ke, int t) {
    // TN: a(m, k) = A[k lda + m]; NT: b(k, n) = B[n ldb + k]
    if constexpr (BF3) {
        fetch_bf3<OP == OP_TN, TM>(st.a, A, lda, M, m0, k0, ke, t);
        fetch_bf3<OP != OP_NT, TN>(st.b, B, ldb, N, n0, k0, ke, t);
    } else {
        fetch_f32<OP == OP_TN, TM>(st.a, A, lda, M, m0, k0, ke, t);
        fetch_f32<OP != OP_NT, TN>(st.b, B, ldb, N, n0, k0, ke, t);
    }
}

template <int OP, int TM, int TN, bool BF3>
__device__ __forceinline__ void gemm_stash(const Stage<TM, TN> &st, float *As, float *Bs, int t) {
    if constexpr (BF3) {
        stash_bf3<OP == OP_TN, TM>(st.a, reinterpret_cast<uint16_t *>(As), t);
        stash_bf3<OP != OP_NT, TN>(st.b, reinterpret_cast<uint16_t *>(Bs), t);
    } else {
        stash_f32<OP == OP_TN, TM>(st.a, As, t);
        stash_f32<OP != OP_NT, TN>(st.b, Bs, t);
    }
}

// C[m][n] = sum_k a(m, k) b(k, n) over k in [k_begin(z), k_end(z)), where
//   NN: a(m, k) = A[m lda + k],  b(k, n) = B[k ldb + n]
//   TN: a(m, k) = A[k lda + m],  b(k, n) = B[k ldb + n]
//   NT: a(m, k) = A[m lda + k],  b(k, n) = B[n ldb + k]
// Output tile TM x TN (launched as 32 x 32, 32 x 64 or 64 x 64); each of the four waves
// computes a TM/2 x TN/2 quarter as (TM/32) x (TN/32) MFMA tiles of 16 x 16.
// Grid: (ceil(M/TM), ceil(N/TN), splits); split z covers k in [z kc, min(K,
// z kc + kc)) and writes C + z * c_split. N and the contiguous dimension of
// every operand are multiples of 16 (hidden widths and d_in); M and K are
// arbitrary.
struct GemmArgs {
    const float *A;
    int lda;
    const float *B;
    int ldb;
    float *C;
    int ldc;
    int64_t c_split, M;
    int N;
    int64_t K, kc;
    const float *G;   // mask operand of the MASK epilogues
    int ldg;
    int gx, gy, gz;   // grid of this product, in tiles
    // MASK_DW1: the layer's input rows X [M x D_IN] and where row tile bx
    // writes its partial of dW_1 ([D_IN x N] at dw1 + bx * dw1_split)
    const float *X;
    float *dw1;
    int64_t dw1_split;
};

// LDS floats of one workgroup of a TM x TN product (two buffers of each operand)
__host__ __device__ constexpr int gemm_lds_floats(int TM, int TN, bool bf3) {
    return 2 * (tile_floats(TM, bf3) + tile_floats(TN, bf3));
}

// The MASK_DW1 epilogue's second half: the workgroup's tile of G_1 (rows
// [m0, m0 + TM) of the batch, units [n0, n0 + TN); masked, in g, rows past M
// zero) times the same rows of X gives that row tile's partial of
// dW_1 = X^T G_1 (eq. 18 at the first layer) for those units, a sum over the
// tile's TM rows in a fixed order. Both operands go through LDS (the K loop is
// done with it); the product is TM / 4 steps of v_mfma_f32_16x16x4f32 per 16 x 16
// output tile, two output tiles per wave (D_IN = 32 inputs x TN = 64 units).
template <int TM, int TN, int MI, int NJ>
__device__ __forceinline__ void dw1_partial(const GemmArgs &g, int bx, int by, const f4 (&gt)[MI][NJ],
                                            float *__restrict__ lds) {
    static_assert(TN == 64 && D_IN == 32, "dW_1 partial tile");
    constexpr int XS = D_IN + 1, GS = TN + 1;   // LDS row strides (floats)
    float *Xs = lds, *Gs = lds + TM * XS;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, lq = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)bx * TM;
    __syncthreads();   // every wave is done with the K loop's LDS
#pragma unroll
    for (int e = t; e < TM * D_IN; e += 256) {
        const int r = e / D_IN, k = e % D_IN;
        const int64_t m = m0 + r;
        Xs[r * XS + k] = m < g.M ? g.X[m * D_IN + k] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                Gs[(wm * (TM / 2) + i * 16 + 4 * lq + v) * GS + wn * (TN / 2) + j * 16 + li] = gt[i][j][v];
    __syncthreads();
    // wave w: inputs 16 (w & 1) .. + 15, units 32 (w >> 1) .. + 31 (two tiles)
    const int it = wave & 1, ub = (wave >> 1) * 32;
    f4 p[2] = {f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < TM / 4; ++ks) {
        const int r = 4 * ks + lq;
        const float a = Xs[r * XS + 16 * it + li];
#pragma unroll
        for (int u = 0; u < 2; ++u)
            p[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Gs[r * GS + ub + 16 * u + li], p[u], 0, 0, 0);
    }
    // lane (li, lq) holds P[input 16 it + 4 lq + v][unit ub + 16 u + li]
    float *dst = g.dw1 + (int64_t)bx * g.dw1_split + (int64_t)by * TN;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v)
            dst[(int64_t)(16 * it + 4 * lq + v) * g.N + ub + 16 * u + li] = p[u][v];
}

// One output tile (bx, by) of split bz; lds holds gemm_lds_floats(TM, TN, BF3).
template <int OP, int EP, int TM, int TN, bool BF3>
__device__ __forceinline__ void gemm_block(const GemmArgs &g, int bx, int by, int bz,
                                           float *__restrict__ lds) {
    constexpr int MI = TM / 32, NJ = TN / 32;   // 16 x 16 MFMA tiles per wave
    constexpr int AS = kmajor_stride(TM), BS = kmajor_stride(TN);
    float *As2[2] = {lds, lds + tile_floats(TM, BF3)};
    float *Bs2[2] = {lds + 2 * tile_floats(TM, BF3), lds + 2 * tile_floats(TM, BF3) + tile_floats(TN, BF3)};
    const float *__restrict__ A = g.A;
    const float *__restrict__ B = g.B;
    const float *__restrict__ G = g.G;
    const int lda = g.lda, ldb = g.ldb, ldg = g.ldg, ldc = g.ldc, N = g.N;
    const int64_t M = g.M, K = g.K, kc = g.kc;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, lq = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)bx * TM;
    const int n0 = by * TN;
    const int64_t kb = (int64_t)bz * kc;
    const int64_t ke = kb + kc < K ? kb + kc : K;

    // acc: the products (fp32) or the leading part products a0 b0 (bf16x3);
    // lo: the other five part products (bf16x3 only)
    f4 acc[MI][NJ], lo[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = lo[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    // NS chunks in flight: chunk c + NS is fetched into the registers chunk c
    // has just left, while chunk c is on the matrix cores. Chunks alternate
    // between two LDS buffers, so one barrier per chunk suffices: the buffer a
    // chunk is written to was last read by the chunk before the previous
    // barrier, which every wave has passed. Every pass of the main loop issues
    // the same loads (the fetches past the last chunk read the zero block and
    // are never stashed), so the compiler can wait for each stage's own loads
    // only, not for all loads in flight.
    constexpr int NS = GSTAGES;
    const int64_t nch = (ke - kb + GK - 1) / GK;
    Stage<TM, TN> st[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q)
        gemm_fetch<OP, TM, TN, BF3>(st[q], A, lda, B, ldb, M, N, m0, n0, kb + q * GK, ke, t);
    // the mask of the epilogue, loaded now (clamped addresses, no lane condition)
    // so that its loads overlap the K loop instead of each waiting at the end
    constexpr bool MASKED = EP == EP_MASK || EP == EP_MASK_DW1;
    float gm[MASKED ? MI : 1][MASKED ? NJ : 1][4];
    if constexpr (MASKED) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const int n = n0 + wn * (TN / 2) + j * 16 + li;
                const int nc = n < N ? n : N - 1;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t m = m0 + wm * (TM / 2) + i * 16 + 4 * lq + v;
                    gm[i][j][v] = G[(m < M ? m : M - 1) * ldg + nc];
                }
            }
    }
    // fp32: eight k steps of 4 on the matrix cores.
    // bf16x3: lane (li, lq) reads k in [8 lq, 8 lq + 8) of row li of each 16-row
    // operand tile, for every part. The leading part product a0 b0 accumulates
    // in acc, the five smaller ones (below 2^-7 |a b| together) in lo, smallest
    // first, so that their roundings are relative to their own sum, not to the
    // whole dot product. The B parts are read once per chunk and the A parts
    // one row tile at a time (the registers of three workgroups per CU); each
    // part pair's products of a row tile go out back to back (independent
    // accumulators).
    auto mfma_chunk = [&](int buf) __attribute__((always_inline)) {
        if constexpr (BF3) {
            const uint16_t *As = reinterpret_cast<const uint16_t *>(As2[buf]);
            const uint16_t *Bs = reinterpret_cast<const uint16_t *>(Bs2[buf]);
            u4v b[NJ][3];
#pragma unroll
            for (int p = 0; p < 3; ++p)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    b[j][p] = *reinterpret_cast<const u4v *>(
                        Bs + (p * TN + wn * (TN / 2) + j * 16 + li) * GK + swz(li, 8 * lq));
            constexpr int PA[5] = {2, 1, 0, 1, 0}, PB[5] = {0, 1, 2, 0, 1};
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                u4v a[3];
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    a[p] = *reinterpret_cast<const u4v *>(
                        As + (p * TM + wm * (TM / 2) + i * 16 + li) * GK + swz(li, 8 * lq));
#pragma unroll
                for (int q = 0; q < 5; ++q)
#pragma unroll
                    for (int j = 0; j < NJ; ++j) lo[i][j] = mfma_bf16(a[PA[q]], b[j][PB[q]], lo[i][j]);
#pragma unroll
                for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_bf16(a[0], b[j][0], acc[i][j]);
            }
        } else {
            const float *As = As2[buf], *Bs = Bs2[buf];
#pragma unroll
            for (int ks = 0; ks < GK / 4; ++ks) {
                const int kr = ks * 4 + lq;
                float a[MI], b[NJ];
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int m = wm * (TM / 2) + i * 16 + li;
                    a[i] = OP == OP_TN ? As[kr * AS + m] : As[m * GMS + kr];
                }
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const int n = wn * (TN / 2) + j * 16 + li;
                    b[j] = OP == OP_NT ? Bs[n * GMS + kr] : Bs[kr * BS + n];
                }
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
            }
        }
    };
    int64_t c = 0;
    for (; c + NS <= nch; c += NS) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const int buf = (int)((c + q) & 1);
            gemm_stash<OP, TM, TN, BF3>(st[q], As2[buf], Bs2[buf], t);
            __syncthreads();
            gemm_fetch<OP, TM, TN, BF3>(st[q], A, lda, B, ldb, M, N, m0, n0, kb + (c + q + NS) * GK, ke, t);
            mfma_chunk(buf);
        }
    }
    // the last nch - c < NS chunks, already in registers
#pragma unroll
    for (int q = 0; q < NS - 1; ++q) {
        if (c + q < nch) {
            const int buf = (int)((c + q) & 1);
            gemm_stash<OP, TM, TN, BF3>(st[q], As2[buf], Bs2[buf], t);
            __syncthreads();
            mfma_chunk(buf);
        }
    }
    // ---- epilogue: lane holds C[4 lq + v][li] of each 16 x 16 tile ----
    float *Cz = g.C + (int64_t)bz * g.c_split;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int n = n0 + wn * (TN / 2) + j * 16 + li;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * (TM / 2) + i * 16 + 4 * lq + v;
                if (m >= M || n >= N) {
                    if constexpr (EP == EP_MASK_DW1) acc[i][j][v] = 0.0f;   // no row: no term
                    continue;
                }
                float r = BF3 ? acc[i][j][v] + lo[i][j][v] : acc[i][j][v];
                // eq. 12; a NaN passes (a diverged step must reach the loss: an
                // infinite operand leaves NaN in its split parts)
                if constexpr (EP == EP_RELU) r = r <= 0.0f ? 0.0f : r;
                if constexpr (MASKED) r = gm[i][j][v] > 0.0f ? r : 0.0f;    // eq. 17
                if constexpr (EP == EP_MASK_DW1) acc[i][j][v] = r;
                Cz[m * ldc + n] = r;
            }
        }
    if constexpr (EP == EP_MASK_DW1) dw1_partial<TM, TN, MI, NJ>(g, bx, by, acc, lds);
}

// The bf16x3 tiles are compiled for three workgroups per CU (the most their LDS
// allows; about 168 registers a lane), the fp32 ones without a bound.
template <int OP, int EP, int TM, int TN, bool BF3>
__global__ __launch_bounds__(256, BF3 ? 3 : 1) void k_gemm(const GemmArgs g) {
    __shared__ __attribute__((aligned(16))) float lds[gemm_lds_floats(TM, TN, BF3)];
    gemm_block<OP, EP, TM, TN, BF3>(g, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

// Two independent products in one launch (a one-dimensional grid): blocks
// [0, g1.gx g1.gy g1.gz) compute the first, the rest the second. With both
// resident together the CUs hold twice the workgroups of either alone.
template <int OP1, int EP1, int TM1, int TN1, int OP2, int EP2, int TM2, int TN2, bool BF3>
__global__ __launch_bounds__(256, BF3 ? 3 : 1) void k_gemm_pair(const GemmArgs g1, const GemmArgs g2) {
    constexpr int L1 = gemm_lds_floats(TM1, TN1, BF3), L2 = gemm_lds_floats(TM2, TN2, BF3);
    __shared__ __attribute__((aligned(16))) float lds[L1 > L2 ? L1 : L2];
    const int n1 = g1.gx * g1.gy * g1.gz;
    int b = blockIdx.x;
    if (b < n1) {
        gemm_block<OP1, EP1, TM1, TN1, BF3>(g1, b % g1.gx, (b / g1.gx) % g1.gy, b / (g1.gx * g1.gy), lds);
    } else {
        b -= n1;
        gemm_block<OP2, EP2, TM2, TN2, BF3>(g2, b % g2.gx, (b / g2.gx) % g2.gy, b / (g2.gx * g2.gy), lds);
    }
}

// Xb[t][k] = X[r_t][k], Yb[t] = Y[r_t], r_t = idx[off + t] (or off + t);
// out-of-range rows read row 0 and raise the sticky error.
struct GatherArgs {
    const float *X, *Y;
    int64_t n_rows;
    const int32_t *idx;
    int64_t off, nb;
    float *Xb, *Yb;
    int32_t *err;
};

// Element e of the gather: float4 e % 8 of batch row e / 8.
__device__ __forceinline__ void gather_one(const GatherArgs &g, int64_t e) {
    if (e >= g.nb * (D_IN / 4)) return;
    const int64_t t = e / (D_IN / 4);
    const int q = (int)(e % (D_IN / 4));
    int64_t r = g.idx ? (int64_t)g.idx[g.off + t] : g.off + t;
    if (r < 0 || r >= g.n_rows) {
        __hip_atomic_store(g.err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r = 0;
    }
    reinterpret_cast<float4 *>(g.Xb)[t * (D_IN / 4) + q] =
        reinterpret_cast<const float4 *>(g.X)[r * (D_IN / 4) + q];
    if (q == 0) g.Yb[t] = g.Y ? g.Y[r] : 0.0f;
}

__global__ __launch_bounds__(256) void k_deep_gather(const GatherArgs g) {
    gather_one(g, (int64_t)blockIdx.x * 256 + threadIdx.x);
}

// Forward output, one wave per row: Ypred = H_L w_o (eq. 13).
__global__ __launch_bounds__(256) void k_deep_ypred(const float *__restrict__ H, int h,
                                                    const float *__restrict__ wo, int64_t nb,
                                                    float *__restrict__ ypred) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= nb) return;
    const float *hr = H + r * h;
    float s = 0.0f;
    for (int j = lane; j < h; j += 64) s = fmaf(hr[j], wo[j], s);
    s = sum64(s);
    if (lane == 0) ypred[r] = s;
}

// Output layer of a training step over row chunk z = blockIdx.x (rows [z kc,
// min(nb, z kc + kc))); wave w of OUT_W takes rows w, w + OUT_W, ... of the chunk and lane l
// units l, l + 64, ... (HU of them). Per row: Ypred = H_L w_o (eq. 13),
// r = Ypred - Y, r^2, dZ_o = (2/n_b) r (eq. 15) and G_L = dZ_o w_o^T (.)
// [H_L > 0] (eq. 17); each lane also sums H_L[r][j] dZ_o[r] over its rows in
// row order (eq. 16), and the OUT_W waves' sums are added in wave order into
// the chunk's dw_o partial. A wave loads OUT_R rows before it reduces any of
// them, so that their loads are in flight together.
constexpr int OUT_R = 4;
constexpr int OUT_W = 8;                   // waves per workgroup of the output kernel
constexpr int OUT_ROWS = OUT_W * OUT_R;    // rows of one output-kernel pass (chunk granule)
template <int HU>
__global__ __launch_bounds__(64 * OUT_W) void k_deep_out(const float *__restrict__ H, int h,
                                                  const float *__restrict__ wo,
                                                  const float *__restrict__ Yb, int64_t nb,
                                                  int64_t kc, float scale, float *__restrict__ sq,
                                                  float *__restrict__ Gout,
                                                  float *__restrict__ dwo_part) {
    __shared__ float wsum[OUT_W][64 * HU];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t rb = (int64_t)blockIdx.x * kc;
    const int64_t re = rb + kc < nb ? rb + kc : nb;
    float wov[HU], acc[HU];
#pragma unroll
    for (int i = 0; i < HU; ++i) {
        wov[i] = wo[lane + 64 * i];
        acc[i] = 0.0f;
    }
    for (int64_t r0 = rb + wave; r0 < re; r0 += OUT_W * OUT_R) {
        // rows past the chunk load its last row and are dropped below
        float hv[OUT_R][HU], yv[OUT_R];
#pragma unroll
        for (int j = 0; j < OUT_R; ++j) {
            const int64_t r = r0 + OUT_W * j < re ? r0 + OUT_W * j : re - 1;
            const float *hr = H + r * h;
#pragma unroll
            for (int i = 0; i < HU; ++i) hv[j][i] = hr[lane + 64 * i];
            yv[j] = Yb[r];
        }
#pragma unroll
        for (int j = 0; j < OUT_R; ++j) {
            const int64_t r = r0 + OUT_W * j;
            float s = 0.0f;
#pragma unroll
            for (int i = 0; i < HU; ++i) s = fmaf(hv[j][i], wov[i], s);
            s = sum64(s);
            if (r >= re) continue;
            const float res = s - yv[j];
            const float g = scale * res;
            if (lane == 0) sq[r] = res * res;
            float *gr = Gout + r * h;
#pragma unroll
            for (int i = 0; i < HU; ++i) {
                gr[lane + 64 * i] = hv[j][i] > 0.0f ? g * wov[i] : 0.0f;
                acc[i] = fmaf(hv[j][i], g, acc[i]);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < HU; ++i) wsum[wave][lane + 64 * i] = acc[i];
    __syncthreads();
    for (int j = threadIdx.x; j < h; j += 64 * OUT_W) {
        float v = wsum[0][j];
#pragma unroll
        for (int w = 1; w < OUT_W; ++w) v += wsum[w][j];
        dwo_part[(int64_t)blockIdx.x * h + j] = v;
    }
}

// Row-chunk split of each parameter segment's gradient (W_1 .. W_L, then w_o).
// Segment s keeps its chunk partials at part + part_off[s], chunk z at
// z * size(s).
struct SplitPlan {
    int nseg;
    int64_t seg_end[DEEP_MAX_LAYERS + 1];   // exclusive end of segment s in the flat array
    int splits[DEEP_MAX_LAYERS + 1];        // row chunks (partials) of segment s
    int64_t kc[DEEP_MAX_LAYERS + 1];        // rows per chunk
    int64_t part_off[DEEP_MAX_LAYERS + 1];  // offset of segment s's partials
};

// Sum the chunk partials of every parameter's gradient in chunk order, then
// eq. 19 (sgd) or write the gradient: workgroups [0, napply). Workgroup napply
// reduces the batch loss instead (eq. 14): thread i sums rows i, i + 256, ...,
// then a fixed binary tree; step and epoch loss as in the one-layer paths. The
// workgroups after it gather the next training step's rows (the gathered
// buffers' last readers, the W_1 gradient and the output kernel, ran before).
__global__ __launch_bounds__(256) void k_deep_apply(const float *__restrict__ part, SplitPlan sp,
                                                    int64_t np, int napply, float *__restrict__ params,
                                                    float *__restrict__ dparams, float lr, int sgd,
                                                    const float *__restrict__ sq, int64_t nb,
                                                    ReduceArgs ra, const GatherArgs next) {
    constexpr int U = 32;     // loads of one batch per lane; the adds stay in index order
    if ((int)blockIdx.x > napply) {
        gather_one(next, (int64_t)(blockIdx.x - napply - 1) * 256 + threadIdx.x);
        return;
    }
    if ((int)blockIdx.x == napply) {
        __shared__ float red[256];
        const int i = threadIdx.x;
        float v = 0.0f;
        for (int64_t t0 = i; t0 < nb; t0 += 256 * U) {
            float x[U];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int64_t t = t0 + 256 * j;
                x[j] = sq[t < nb ? t : nb - 1];
            }
#pragma unroll
            for (int j = 0; j < U; ++j)
                if (t0 + 256 * j < nb) v += x[j];
        }
        red[i] = v;
        __syncthreads();
        for (int w = 128; w >= 1; w >>= 1) {
            if (i < w) red[i] += red[i + w];
            __syncthreads();
        }
        if (i == 0) {
            const float sse = red[0];
            const float L = sse * ra.inv_nb;
            flag_nonfinite(sse, &ra.ctl->err);
            if (ra.loss) ra.loss[0] = L;
            if (ra.step_loss) ra.step_loss[ra.step] = L;
            if (ra.epoch_loss) {
                double acc = ra.first_in_epoch ? 0.0 : ra.ctl->epoch_sse;
                acc += (double)sse;
                ra.ctl->epoch_sse = acc;
                ra.epoch_loss[ra.epoch] = (float)(acc * ra.inv_n);
            }
        }
        return;
    }
    // Segment ends are multiples of 64, so a wave lies in one segment: look it
    // up once per wave, in scalar registers.
    const int64_t p0 = __builtin_amdgcn_readfirstlane((int)blockIdx.x * 256 + (int)(threadIdx.x & ~63));
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (p >= np) return;
    int seg = 0;
    while (seg + 1 < sp.nseg && p0 >= sp.seg_end[seg]) ++seg;
    const int64_t start = seg == 0 ? 0 : sp.seg_end[seg - 1];
    const int64_t size = sp.seg_end[seg] - start;
    const int n = sp.splits[seg];
    const float *q = part + sp.part_off[seg] + (p - start);
    const float w = sgd ? params[p] : 0.0f;
    float v = 0.0f;
    int z0 = 0;
    for (; z0 + 2 * U <= n; z0 += 2 * U) {   // two batches of loads in flight, added in order
        float x[U], y[U];
#pragma unroll
        for (int j = 0; j < U; ++j) x[j] = q[(int64_t)(z0 + j) * size];
#pragma unroll
        for (int j = 0; j < U; ++j) y[j] = q[(int64_t)(z0 + U + j) * size];
#pragma unroll
        for (int j = 0; j < U; ++j) v += x[j];
#pragma unroll
        for (int j = 0; j < U; ++j) v += y[j];
    }
    for (; z0 + U <= n; z0 += U) {
        float x[U];
#pragma unroll
        for (int j = 0; j < U; ++j) x[j] = q[(int64_t)(z0 + j) * size];
#pragma unroll
        for (int j = 0; j < U; ++j) v += x[j];
    }
    for (; z0 < n; z0 += 4) {    // the last n mod U partials, four loads at a time
        float x[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int z = z0 + j < n ? z0 + j : n - 1;
            x[j] = q[(int64_t)z * size];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (z0 + j < n) v += x[j];
    }
    if (sgd) params[p] = w - lr * v;
    else dparams[p] = v;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

struct DeepCtx {
    int hidden = 0, layers = 0;
    int64_t max_batch = 0, np = 0;
    float *params = nullptr;
    Control *ctl = nullptr;
    float *Xb = nullptr, *Yb = nullptr, *sq = nullptr;
    float *H = nullptr;       // [layers][max_batch x hidden]
    float *G[2] = {nullptr, nullptr};
    float *part = nullptr;    // gradient partials, segment s at part_off[s] (plan of max_batch)
    int64_t part_off[DEEP_MAX_LAYERS + 1] = {};
    hipStream_t stream = nullptr;
    bool profile = false, ev_valid = false;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
};

static int64_t deep_np(int h, int L) { return (int64_t)D_IN * h + (int64_t)(L - 1) * h * h + h; }
static int64_t layer_offset(int h, int l) {   // W_l, l = 1..L; w_o at l = L + 1
    return l == 1 ? 0 : (int64_t)D_IN * h + (int64_t)(l - 2) * h * h;
}
static size_t pad64f(size_t n) { return (n + 63) / 64 * 64; }

static bool deep_shape_ok(int32_t d_in, int32_t hidden, int32_t layers) {
    return d_in == D_IN && hidden >= 64 && hidden <= 1024 && hidden % 64 == 0 && layers >= 1 &&
           layers <= DEEP_MAX_LAYERS;
}

// Row chunks of segment s's gradient before rounding the chunk length: a weight
// segment W_l gets enough chunks for its GEMM to reach about 256 workgroups
// (output tiles x chunks) at h <= 256 and 512 above, at most SPLIT_MAX, with at
// least 64 rows a chunk (at h = 256 and batch 4096: 16 chunks of 256 rows, the
// back-propagation's K, so both products of a pair run eight K chunks); w_o
// gets one chunk per OUT_ROWS rows of the output kernel, at most OUT_CHUNKS_MAX. This
// count never falls as nb grows, and the chunks a plan uses never exceed it, so
// the count at max_batch sizes the partial buffer for every batch.
static int64_t seg_chunks(int h, int L, int64_t nb, int s) {
    int64_t splits;
    if (s == 0 && L > 1) {
        // dW_1 comes from the epilogue of the back-propagation into layer 1,
        // one partial per row tile of that product (32 or 64 rows)
        splits = (nb + 31) / 32;
    } else if (s < L) {
        const int64_t K = s == 0 ? D_IN : h;
        const int64_t tiles = ((K + GT - 1) / GT) * (h / GT);
        const int64_t target = h <= 256 ? 256 : 512;
        splits = (target + tiles - 1) / tiles;
        const int64_t by_rows = (nb + 63) / 64;
        if (splits > by_rows) splits = by_rows;
        splits = splits > SPLIT_MAX ? SPLIT_MAX : splits;
    } else {
        splits = (nb + OUT_ROWS - 1) / OUT_ROWS;
        splits = splits > OUT_CHUNKS_MAX ? OUT_CHUNKS_MAX : splits;
    }
    return splits < 1 ? 1 : splits;
}

static int64_t seg_size(int h, int L, int s) { return s < L ? (s == 0 ? D_IN : h) * (int64_t)h : h; }

// Offsets of each segment's partials for batches up to mb (packed).
static int64_t part_layout(int h, int L, int64_t mb, int64_t *off) {
    int64_t o = 0;
    for (int s = 0; s <= L; ++s) {
        if (off) off[s] = o;
        o += pad64f((size_t)(seg_chunks(h, L, mb, s) * seg_size(h, L, s)));
    }
    return o;
}

// The plan of a batch of nb rows: chunk length rounded up to the GEMM's K chunk
// (to the output kernel's pass for w_o), and the chunk count that length gives
// (never more than seg_chunks).
// dw1_rows: with more than one layer, the rows of one back-propagation tile
// into layer 1, whose epilogue writes one dW_1 partial per row tile.
static void split_plan(int h, int L, int64_t nb, const int64_t *part_off, int dw1_rows, SplitPlan *sp) {
    sp->nseg = L + 1;
    for (int s = 0; s <= L; ++s) {
        const int64_t splits = seg_chunks(h, L, nb, s);
        int64_t c = (nb + splits - 1) / splits;
        const int64_t q = s < L ? GK : OUT_ROWS;
        c = (c + q - 1) / q * q;
        if (s == 0 && L > 1) c = dw1_rows;
        sp->kc[s] = c;
        sp->splits[s] = (int)((nb + c - 1) / c);
        sp->seg_end[s] = s < L ? layer_offset(h, s + 2) : deep_np(h, L);
        sp->part_off[s] = part_off[s];
    }
}

static int64_t part_floats(int h, int L, int64_t nb) { return part_layout(h, L, nb, nullptr); }

static size_t deep_ws_floats(int h, int L, int64_t mb) {
    const size_t b = (size_t)mb;
    return pad64f(CTL_BYTES / 4) + pad64f(b * D_IN) + 2 * pad64f(b) +
           (size_t)(L + 2) * pad64f(b * (size_t)h) + (size_t)part_floats(h, L, mb);
}

// Tile choice: 64 x 64, or 32 x 64 where 64-row tiles would leave fewer than
// two workgroups per CU (the 256-wide layers) or M itself is 32 (the weight
// gradient of W_1); a single product (not a pair) narrows that to 32 x 32 where
// it would still leave fewer than four. Larger tiles (128 x 64, 128 x 128) halve the operand
// traffic per MFMA but leave one or two workgroups per CU on the 1024-wide
// products, which measured 6-8 % slower than four. The 64 x 64 tiles (the
// MFMA-heavy products of wide layers) run the bf16x3 flavour, the narrower
// ones (latency-bound, few chunks each) the fp32 one: bf16x3 made the 1024-wide
// net 8 % faster and the 256-wide ones 3-6 % slower.
static GemmArgs gemm_args(const float *A, int lda, const float *B, int ldb, float *C, int ldc,
                          int64_t c_split, int64_t M, int N, int64_t K, int splits, int64_t kc,
                          const float *G, int ldg, bool *small) {
    const int64_t tiles64 = ((M + GT - 1) / GT) * ((N + GT - 1) / GT) * splits;
    *small = M <= 32 || tiles64 < 2 * GEMM_CUS;
    const int tm = *small ? 32 : GT;
    GemmArgs g;
    g.A = A;
    g.lda = lda;
    g.B = B;
    g.ldb = ldb;
    g.C = C;
    g.ldc = ldc;
    g.c_split = c_split;
    g.M = M;
    g.N = N;
    g.K = K;
    g.kc = kc;
    g.G = G;
    g.ldg = ldg;
    g.X = nullptr;
    g.dw1 = nullptr;
    g.dw1_split = 0;
    g.gx = (int)((M + tm - 1) / tm);
    g.gy = (N + GT - 1) / GT;
    g.gz = splits;
    return g;
}

template <int OP, int EP>
static hipError_t gemm(hipStream_t st, const float *A, int lda, const float *B, int ldb, float *C,
                       int ldc, int64_t c_split, int64_t M, int N, int64_t K, int splits,
                       int64_t kc, const float *G = nullptr, int ldg = 0) {
    bool small;
    const GemmArgs g = gemm_args(A, lda, B, ldb, C, ldc, c_split, M, N, K, splits, kc, G, ldg, &small);
    const dim3 grid((unsigned)g.gx, (unsigned)g.gy, (unsigned)g.gz);
    if (small && (int64_t)g.gx * g.gy * g.gz < 4 * GEMM_CUS) {
        // 32 x 32 tiles where 32 x 64 ones would leave fewer than four
        // workgroups per CU
        GemmArgs gn = g;
        gn.gy = (N + 31) / 32;
        hipLaunchKernelGGL((k_gemm<OP, EP, 32, 32, false>), dim3((unsigned)gn.gx, (unsigned)gn.gy, (unsigned)gn.gz),
                           dim3(256), 0, st, gn);
    } else if (small)
        hipLaunchKernelGGL((k_gemm<OP, EP, 32, GT, false>), grid, dim3(256), 0, st, g);
    else
        hipLaunchKernelGGL((k_gemm<OP, EP, GT, GT, true>), grid, dim3(256), 0, st, g);
    return hipGetLastError();
}

// The two independent products g1 (OP1, EP1) and g2 (OP2, EP2) in one launch.
template <int OP1, int EP1, int OP2, int EP2>
static hipError_t gemm_pair(hipStream_t st, const GemmArgs &g1, bool small1, const GemmArgs &g2,
                            bool small2) {
    const dim3 grid((unsigned)(g1.gx * g1.gy * g1.gz + g2.gx * g2.gy * g2.gz));
    if (small1 && small2)
        hipLaunchKernelGGL((k_gemm_pair<OP1, EP1, 32, GT, OP2, EP2, 32, GT, false>), grid, dim3(256), 0, st, g1, g2);
    else if (small1)
        hipLaunchKernelGGL((k_gemm_pair<OP1, EP1, 32, GT, OP2, EP2, GT, GT, false>), grid, dim3(256), 0, st, g1, g2);
    else if (small2)
        hipLaunchKernelGGL((k_gemm_pair<OP1, EP1, GT, GT, OP2, EP2, 32, GT, false>), grid, dim3(256), 0, st, g1, g2);
    else
        hipLaunchKernelGGL((k_gemm_pair<OP1, EP1, GT, GT, OP2, EP2, GT, GT, true>), grid, dim3(256), 0, st, g1, g2);
    return hipGetLastError();
}

#define DEEP_TRY(x)                        \
    do {                                   \
        hipError_t e_ = (x);               \
        if (e_ != hipSuccess) return e_;   \
    } while (0)

static unsigned blocks_of(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Forward of nb gathered rows (Xb) through every hidden layer into c.H.
static hipError_t deep_forward_layers(const DeepCtx &c, int64_t nb) {
    const int h = c.hidden;
    const float *in = c.Xb;
    int K = D_IN;
    for (int l = 1; l <= c.layers; ++l) {
        float *out = c.H + (int64_t)(l - 1) * c.max_batch * h;
        DEEP_TRY((gemm<OP_NN, EP_RELU>(c.stream, in, K, c.params + layer_offset(h, l), h, out, h,
                                       0, nb, h, K, 1, K)));
        in = out;
        K = h;
    }
    return hipSuccess;
}

// The training output kernel, instantiated for h / 64 units per lane.
static hipError_t launch_out(const DeepCtx &c, const float *HL, const float *wo, int64_t nb,
                             int64_t kc, int chunks, float *dwo_part) {
    const float scale = 2.0f / (float)nb;   // eq. 15
    switch (c.hidden / 64) {
#define DEEP_OUT_CASE(U)                                                                          \
    case U:                                                                                       \
        hipLaunchKernelGGL((k_deep_out<U>), dim3(chunks), dim3(64 * OUT_W), 0, c.stream, HL, c.hidden, wo, \
                           c.Yb, nb, kc, scale, c.sq, c.G[0], dwo_part);                           \
        return hipGetLastError();
        DEEP_OUT_CASE(1) DEEP_OUT_CASE(2) DEEP_OUT_CASE(3) DEEP_OUT_CASE(4)
        DEEP_OUT_CASE(5) DEEP_OUT_CASE(6) DEEP_OUT_CASE(7) DEEP_OUT_CASE(8)
        DEEP_OUT_CASE(9) DEEP_OUT_CASE(10) DEEP_OUT_CASE(11) DEEP_OUT_CASE(12)
        DEEP_OUT_CASE(13) DEEP_OUT_CASE(14) DEEP_OUT_CASE(15) DEEP_OUT_CASE(16)
#undef DEEP_OUT_CASE
    }
    return hipErrorInvalidValue;
}

static GatherArgs gather_args(const DeepCtx &c, const float *X, const float *Y, int64_t n_rows,
                              const int32_t *idx, int64_t off, int64_t nb) {
    GatherArgs g;
    g.X = X;
    g.Y = Y;
    g.n_rows = n_rows;
    g.idx = idx;
    g.off = off;
    g.nb = nb;
    g.Xb = c.Xb;
    g.Yb = c.Yb;
    g.err = &c.ctl->err;
    return g;
}

// One step (or one gradient evaluation) on batch rows [off, off + nb) of idx.
// With gathered, the rows are already in Xb / Yb (gathered by the previous
// step's update kernel); with next, the update kernel also gathers the rows of
// the next step.
static hipError_t deep_step(DeepCtx &c, const float *X, int64_t n_rows, const float *Y,
                            const int32_t *idx, int64_t off, int64_t nb, const ReduceArgs &ra,
                            float *dparams, bool gathered = false, const GatherArgs *next = nullptr) {
    const int h = c.hidden, L = c.layers;
    const int64_t mbh = c.max_batch * h;
    if (!gathered) {
        hipLaunchKernelGGL(k_deep_gather, dim3(blocks_of(nb * (D_IN / 4), 256)), dim3(256), 0,
                           c.stream, gather_args(c, X, Y, n_rows, idx, off, nb));
        DEEP_TRY(hipGetLastError());
    }
    DEEP_TRY(deep_forward_layers(c, nb));
    const float *HL = c.H + (int64_t)(L - 1) * mbh;
    const float *wo = c.params + layer_offset(h, L + 1);
    int cur = 0;
    // with more than one layer, dW_1 comes from the epilogue of the
    // back-propagation into layer 1 (one partial per row tile of that product)
    int dw1_rows = 0;
    if (L > 1) {
        bool small;
        (void)gemm_args(c.G[0], h, c.params, h, c.G[1], h, 0, nb, h, h, 1, h, c.Xb, h, &small);
        dw1_rows = small ? 32 : GT;
    }
    SplitPlan sp;
    split_plan(h, L, nb, c.part_off, dw1_rows, &sp);
    // output layer: r^2, G_L and the dw_o partials of each row chunk
    DEEP_TRY(launch_out(c, HL, wo, nb, sp.kc[L], sp.splits[L], c.part + sp.part_off[L]));
    for (int l = L; l >= 1; --l) {
        const int K = l == 1 ? D_IN : h;
        const float *Hin = l == 1 ? c.Xb : c.H + (int64_t)(l - 2) * mbh;
        // dW_l = H_{l-1}^T G_l, eq. 18, split over row chunks
        bool s1, s2;
        const GemmArgs gw = gemm_args(Hin, K, c.G[cur], h, c.part + sp.part_off[l - 1], h,
                                      (int64_t)K * h, K, h, nb, sp.splits[l - 1], sp.kc[l - 1],
                                      nullptr, 0, &s1);
        if (l > 1) {
            // G_{l-1} = (G_l W_l^T) (.) [H_{l-1} > 0], eq. 17 one layer down; it
            // reads G_l as the weight gradient does and writes the other buffer,
            // so the two products share one launch. Into layer 1 (l = 2) its
            // epilogue also forms the row tile's partial of dW_1 = X^T G_1.
            GemmArgs gg = gemm_args(c.G[cur], h, c.params + layer_offset(h, l), h, c.G[cur ^ 1], h,
                                    0, nb, h, h, 1, h, Hin, h, &s2);
            if (l == 2) {
                gg.X = c.Xb;
                gg.dw1 = c.part + sp.part_off[0];
                gg.dw1_split = (int64_t)D_IN * h;
                DEEP_TRY((gemm_pair<OP_TN, EP_NONE, OP_NT, EP_MASK_DW1>(c.stream, gw, s1, gg, s2)));
            } else {
                DEEP_TRY((gemm_pair<OP_TN, EP_NONE, OP_NT, EP_MASK>(c.stream, gw, s1, gg, s2)));
            }
            cur ^= 1;
        } else if (L == 1) {
            DEEP_TRY((gemm<OP_TN, EP_NONE>(c.stream, Hin, K, c.G[cur], h, c.part + sp.part_off[l - 1], h,
                                           (int64_t)K * h, K, h, nb, sp.splits[l - 1], sp.kc[l - 1])));
        }
    }
    // every gradient's partials summed and applied; the last workgroup takes the loss
    const unsigned napply = blocks_of(c.np, 256);
    GatherArgs none;
    memset(&none, 0, sizeof(none));
    const unsigned ng = next ? blocks_of(next->nb * (D_IN / 4), 256) : 0;
    hipLaunchKernelGGL(k_deep_apply, dim3(napply + 1 + ng), dim3(256), 0, c.stream, c.part, sp,
                       c.np, (int)napply, c.params, dparams, ra.lr, ra.sgd, c.sq, nb, ra,
                       next ? *next : none);
    return hipGetLastError();
}

}  // namespace mlp

using namespace mlp;

struct mlp_deep_ctx : mlp::DeepCtx {};

extern "C" int64_t mlp_deep_param_count(int32_t d_in, int32_t hidden, int32_t layers) {
    if (!deep_shape_ok(d_in, hidden, layers)) return 0;
    return deep_np(hidden, layers);
}

extern "C" size_t mlp_deep_workspace_bytes(int32_t d_in, int32_t hidden, int32_t layers,
                                           int64_t max_batch) {
    if (!deep_shape_ok(d_in, hidden, layers) || max_batch < 1 || max_batch > MLP_MAX_BATCH) return 0;
    return sizeof(float) * deep_ws_floats(hidden, layers, max_batch);
}

extern "C" mlp_status mlp_deep_init(mlp_deep_t *out, int32_t d_in, int32_t hidden, int32_t layers,
                                    int32_t d_out, int64_t max_batch, float *params,
                                    void *workspace, size_t ws_bytes, void *stream) {
    if (!out || !params || !workspace) return MLP_ERR_INVALID_ARG;
    if (!deep_shape_ok(d_in, hidden, layers) || d_out != 1) return MLP_ERR_UNSUPPORTED;
    if (max_batch < 1 || max_batch > MLP_MAX_BATCH) return MLP_ERR_INVALID_ARG;
    if (ws_bytes < mlp_deep_workspace_bytes(d_in, hidden, layers, max_batch) ||
        ((uintptr_t)workspace & 255u))
        return MLP_ERR_WORKSPACE;
    mlp_deep_ctx *c = new (std::nothrow) mlp_deep_ctx();
    if (!c) return MLP_ERR_HIP;
    c->hidden = hidden;
    c->layers = layers;
    c->max_batch = max_batch;
    c->np = deep_np(hidden, layers);
    c->params = params;
    c->stream = (hipStream_t)stream;
    float *p = (float *)workspace;
    auto take = [&](size_t n) {
        float *q = p;
        p += pad64f(n);
        return q;
    };
    const size_t b = (size_t)max_batch, bh = b * (size_t)hidden;
    c->ctl = (Control *)take(CTL_BYTES / 4);
    c->Xb = take(b * D_IN);
    c->Yb = take(b);
    c->sq = take(b);
    c->H = p;
    p += (size_t)layers * pad64f(bh);
    c->G[0] = take(bh);
    c->G[1] = take(bh);
    c->part = take((size_t)part_layout(hidden, layers, max_batch, c->part_off));
    Ctx tmp;
    tmp.ctl = c->ctl;
    tmp.stream = c->stream;
    if (clear_control(tmp) != hipSuccess) {
        delete c;
        return MLP_ERR_HIP;
    }
    *out = c;
    return MLP_OK;
}

extern "C" void mlp_deep_destroy(mlp_deep_t c) {
    if (!c) return;
    if (c->ev0) (void)hipEventDestroy(c->ev0);
    if (c->ev1) (void)hipEventDestroy(c->ev1);
    delete c;
}

static mlp_status deep_status(hipError_t e) { return e == hipSuccess ? MLP_OK : MLP_ERR_HIP; }

extern "C" mlp_status mlp_deep_forward(mlp_deep_t c, const float *X, int64_t n_rows,
                                       const int32_t *idx, int64_t B, float *Ypred) {
    if (!c || !X || !Ypred || B < 1 || n_rows < 1) return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    const int h = c->hidden;
    const float *HL = c->H + (int64_t)(c->layers - 1) * c->max_batch * h;
    const float *wo = c->params + layer_offset(h, c->layers + 1);
    for (int64_t off = 0; off < B; off += c->max_batch) {
        const int64_t nb = B - off < c->max_batch ? B - off : c->max_batch;
        hipLaunchKernelGGL(k_deep_gather, dim3(blocks_of(nb * (D_IN / 4), 256)), dim3(256), 0,
                           c->stream, gather_args(*c, X, nullptr, n_rows, idx, off, nb));
        if (hipGetLastError() != hipSuccess) return MLP_ERR_HIP;
        if (deep_forward_layers(*c, nb) != hipSuccess) return MLP_ERR_HIP;
        hipLaunchKernelGGL(k_deep_ypred, dim3(blocks_of(nb, 4)), dim3(256), 0, c->stream, HL, h, wo,
                           nb, Ypred + off);
        if (hipGetLastError() != hipSuccess) return MLP_ERR_HIP;
    }
    return MLP_OK;
}

static ReduceArgs deep_args(const mlp_deep_ctx *c, int64_t nb) {
    ReduceArgs a;
    memset(&a, 0, sizeof(a));
    a.inv_nb = (float)(1.0 / (double)nb);
    a.ctl = c->ctl;
    return a;
}

extern "C" mlp_status mlp_deep_backward(mlp_deep_t c, const float *X, int64_t n_rows,
                                        const float *Y, const int32_t *idx, int64_t B,
                                        float *dparams, float *loss) {
    if (!c || !X || !Y || !dparams || B < 1 || B > c->max_batch || n_rows < 1)
        return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    ReduceArgs a = deep_args(c, B);
    a.sgd = 0;
    a.loss = loss;
    return deep_status(deep_step(*c, X, n_rows, Y, idx, 0, B, a, dparams));
}

static void deep_prof(mlp_deep_ctx *c, bool begin) {
    if (!c->profile) return;
    if (begin) {
        if (!c->ev0) (void)hipEventCreate(&c->ev0);
        if (!c->ev1) (void)hipEventCreate(&c->ev1);
        (void)hipEventRecord(c->ev0, c->stream);
    } else {
        (void)hipEventRecord(c->ev1, c->stream);
        c->ev_valid = true;
    }
}

extern "C" mlp_status mlp_deep_sgd_step(mlp_deep_t c, const float *X, int64_t n_rows,
                                        const float *Y, const int32_t *idx, int64_t B, float lr,
                                        float *loss) {
    if (!c || !X || !Y || B < 1 || B > c->max_batch || n_rows < 1 || !isfinite(lr))
        return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    ReduceArgs a = deep_args(c, B);
    a.sgd = 1;
    a.lr = lr;
    a.loss = loss;
    deep_prof(c, true);
    const mlp_status st = deep_status(deep_step(*c, X, n_rows, Y, idx, 0, B, a, nullptr));
    deep_prof(c, false);
    return st;
}

extern "C" mlp_status mlp_deep_train_epochs(mlp_deep_t c, const float *X, const float *Y,
                                            int64_t n, int64_t batch, float lr, int32_t epochs,
                                            const int32_t *perm, int64_t max_steps,
                                            float *epoch_loss, float *step_loss) {
    if (!c || !X || !Y || n < 1 || batch < 1 || batch > c->max_batch || epochs < 1 ||
        !isfinite(lr) || max_steps < -1)
        return MLP_ERR_INVALID_ARG;
    if ((int64_t)epochs * n > ((int64_t)1 << 40)) return MLP_ERR_INVALID_ARG;
    Ctx tmp;
    tmp.stream = c->stream;
    hipError_t e = hipSuccess;
    if (epoch_loss) e = fill(tmp, epoch_loss, epochs, 0.0f);
    if (e != hipSuccess) return MLP_ERR_HIP;
    const int64_t spe = (n + batch - 1) / batch;
    const int64_t total = max_steps >= 0 && max_steps < spe * epochs ? max_steps : spe * epochs;
    int64_t step = 0;
    deep_prof(c, true);
    for (int32_t ep = 0; ep < epochs && e == hipSuccess; ++ep) {
        for (int64_t s = 0; s < spe; ++s) {
            if (step >= total) break;
            const int64_t off = s * batch;
            const int64_t nb = n - off < batch ? n - off : batch;
            ReduceArgs a = deep_args(c, nb);
            a.sgd = 1;
            a.lr = lr;
            a.inv_n = (float)(1.0 / (double)n);
            a.step_loss = step_loss;
            a.step = step;
            a.epoch_loss = epoch_loss;
            a.epoch = ep;
            a.first_in_epoch = s == 0;
            const int32_t *ix = perm ? perm + (int64_t)ep * n : nullptr;
            // the next step's rows are gathered by this step's update kernel
            GatherArgs nxt;
            const bool more = step + 1 < total;
            if (more) {
                const int64_t s2 = s + 1 < spe ? s + 1 : 0;
                const int32_t ep2 = s + 1 < spe ? ep : ep + 1;
                const int64_t off2 = s2 * batch;
                nxt = gather_args(*c, X, Y, n, perm ? perm + (int64_t)ep2 * n : nullptr, off2,
                                  n - off2 < batch ? n - off2 : batch);
            }
            e = deep_step(*c, X, n, Y, ix, off, nb, a, nullptr, step > 0, more ? &nxt : nullptr);
            if (e != hipSuccess) break;
            ++step;
        }
    }
    deep_prof(c, false);
    return deep_status(e);
}

extern "C" mlp_status mlp_deep_check_errors(mlp_deep_t c) {
    if (!c) return MLP_ERR_INVALID_ARG;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return MLP_ERR_HIP;
    int32_t err = 0;
    if (hipMemcpy(&err, &c->ctl->err, sizeof(err), hipMemcpyDeviceToHost) != hipSuccess)
        return MLP_ERR_HIP;
    if (err) {
        Ctx tmp;
        tmp.ctl = c->ctl;
        tmp.stream = c->stream;
        if (clear_control(tmp) != hipSuccess || hipStreamSynchronize(c->stream) != hipSuccess)
            return MLP_ERR_HIP;
        return err == MLP_ERR_NONFINITE ? MLP_ERR_NONFINITE : MLP_ERR_INDEX;
    }
    return MLP_OK;
}

extern "C" mlp_status mlp_deep_profile(mlp_deep_t c, int32_t enable) {
    if (!c) return MLP_ERR_INVALID_ARG;
    c->profile = enable != 0;
    c->ev_valid = false;
    return MLP_OK;
}

extern "C" mlp_status mlp_deep_last_kernel_ms(mlp_deep_t c, float *ms) {
    if (!c || !ms || !c->ev_valid) return MLP_ERR_INVALID_ARG;
    if (hipEventSynchronize(c->ev1) != hipSuccess) return MLP_ERR_HIP;
    return deep_status(hipEventElapsedTime(ms, c->ev0, c->ev1));
}
