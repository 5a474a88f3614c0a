// train_persistent.hip -- single-launch fused mini-batch SGD trainer for the
// d-h-1 ReLU/MSE network (paper Sec. III eqs. 11-19, d = 32), for gfx950.
//
// Decomposition (one workgroup per CU, 4 waves each):
//   - the hidden units are split over PX groups of workgroups; each group lives
//     on one XCD (8 XCDs, one L2 each) and owns U = h/PX units;
//   - inside a group, PR workgroups split the rows of every mini-batch (R rows
//     each) and keep the group's W1 slice [32 x U] and W2 slice [U] in registers.
// One SGD step is then:
//   1. stage the step's rows (gathered through the epoch permutation) in LDS;
//   2. Z1 = X W1 on fp32 MFMA (16x16x4); ReLU mask bits and the partial
//      Ypred over the group's units stay in registers (eqs. 11-13);
//   3. exchange A (across XCDs, PX-way): sum the PX partial Ypred of each row in
//      group order -> full Ypred, residual, dZ2 = (2/n_b) r (eqs. 14-15);
//   4. P = X^T (dZ2 (.) [Z1 > 0]) on MFMA over the workgroup's rows; then
//      dW1 = P diag(W2) and dW2_j = sum_k W1_kj P_kj, which equal eqs. 16-18
//      (H_rj = [Z1_rj > 0] sum_k X_rk W1_kj);
//   5. exchange B (inside the XCD, PR-way reduce-scatter): workgroup b sums,
//      in workgroup order, the P columns of the units it owns and applies
//      W -= lr dW to them (eq. 19);
//   6. exchange C (inside the XCD, all-gather): every workgroup of the group
//      reads the updated slice.
// Exchanges use 64-bit words holding (fp32 value, 32-bit step tag). Writers
// never wait; readers poll one word per peer, then load the rest and retry any
// word whose tag is not yet current. Every sum runs in a fixed order, so
// results are bitwise reproducible and identical in every group that computes
// them. No floating-point atomics are used.
//
// Memory scopes: exchange A stores and all exchange loads are device-coherent
// (sc1). Exchanges B and C stay inside one XCD, whose L2 is shared: their
// stores are plain (write-through L1 into the XCD's L2) when every group was
// verified at start-up to sit on one XCD (hardware XCC id); otherwise they are
// device-coherent as well, which is correct for any placement.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

typedef float f4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ unsigned hw_xcc_id() {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v;
}

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

__device__ __forceinline__ uint64_t pack(float v, uint32_t tag) {
    return ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v);
}
__device__ __forceinline__ uint32_t tag_of(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ float val_of(uint64_t w) { return __uint_as_float((uint32_t)w); }

// device-coherent store / load (sc1)
__device__ __forceinline__ void st_dev(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_dev(const uint64_t *p) {
    return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// XCD-local store: plain (lands in the XCD's L2) or device-coherent
__device__ __forceinline__ void st_loc(uint64_t *p, uint64_t v, bool plain) {
    if (plain)
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SINGLETHREAD);
    else
        st_dev(p, v);
}

// Kernel-wide abort flag (set on a spin timeout); polled while waiting.
struct Sync {
    int32_t *abort;      // device word
    int32_t *err;        // sticky error word
    uint64_t deadline;   // s_memrealtime ticks
};

// Wait until the word at p carries tag; returns its value (0 on abort).
__device__ __forceinline__ float wait_word(const uint64_t *p, uint32_t tag, const Sync &s,
                                           bool &aborted) {
    uint32_t spins = 0;
    while (true) {
        uint64_t w = ld_dev(p);
        if (tag_of(w) == tag) return val_of(w);
        if ((++spins & 63u) == 0) {
            if (__hip_atomic_load(s.abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                aborted = true;
                return 0.0f;
            }
            if (now_ticks() > s.deadline) {
                __hip_atomic_store(s.err, (int32_t)MLP_ERR_TIMEOUT_CODE, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(s.abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                aborted = true;
                return 0.0f;
            }
        }
    }
}

// Sum over the 16 lanes of each lane group (lanes 16q..16q+15) with a fixed
// butterfly, so every lane of the group ends with the same value.
__device__ __forceinline__ float sum16(float v) {
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 1, 64);
    return v;
}
__device__ __forceinline__ float sum32(float v) {
    v += __shfl_xor(v, 16, 64);
    return sum16(v);
}

__device__ __forceinline__ int64_t gather_row(const int32_t *__restrict__ perm, int64_t pos,
                                              int64_t n_rows, int32_t *err) {
    int64_t r = perm ? (int64_t)perm[pos] : pos;
    if (r < 0 || r >= n_rows) {
        __hip_atomic_store(err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r = 0;
    }
    return r;
}

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
// Template: NUW = unit tiles (16 units) per wave, RTW = row tiles (16 rows) per wave.
// Waves: WR x WU = 4; wave w takes row tiles {w % WR + i*WR} and unit tiles
// {w / WR + i*WU} of its workgroup.
template <int NUW, int RTW>
__global__ __launch_bounds__(256) void k_train(const TrainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int s_flags[8];   // 0: group x, 1: rank b, 2: plain local stores, 3: abort, 4: active

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lq = lane >> 4, li = lane & 15;   // lane group (0..3) and index in group
    const TrainPlan &p = a.plan;
    const int U = p.U, R = p.R, PR = p.pr, PX = p.px;
    const int WR = p.wr, WU = p.wu;
    const int wr = wave % WR, wu = wave / WR;
    Sync sync{a.abort, a.err, 0};

    // ---- registration: which XCD am I on, and my rank there -------------------
    if (tid == 0) {
        const unsigned x_hw = hw_xcc_id() & 7u;
        const int rank_x = __hip_atomic_fetch_add(&a.reg[x_hw], 1, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        const int rank_g = __hip_atomic_fetch_add(&a.reg[8], 1, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        // start barrier over the whole launch (once per call)
        __hip_atomic_fetch_add(&a.reg[9], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t_end = now_ticks() + a.timeout_ticks;
        int ab = 0;
        while (__hip_atomic_load(&a.reg[9], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) <
               (int)gridDim.x) {
            if (now_ticks() > t_end) {
                __hip_atomic_store(a.err, (int32_t)MLP_ERR_TIMEOUT_CODE, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                ab = 1;
                break;
            }
        }
        // placement check: PR workgroups on each of XCDs 0..PX-1
        bool placed = !a.force_coherent;
        for (int i = 0; i < PX; ++i)
            if (__hip_atomic_load(&a.reg[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != PR)
                placed = false;
        int gx, gb, active;
        if (placed) {
            gx = (int)x_hw;
            gb = rank_x;
            active = gx < PX && gb < PR;
        } else {
            gx = rank_g / PR;
            gb = rank_g % PR;
            active = rank_g < PX * PR;
        }
        s_flags[0] = gx;
        s_flags[1] = gb;
        s_flags[2] = placed ? 1 : 0;
        s_flags[3] = ab;
        s_flags[4] = active;
    }
    __syncthreads();
    const int gx = s_flags[0], gb = s_flags[1];
    const bool plain = s_flags[2] != 0;
    bool aborted = s_flags[3] != 0;
    const bool active = s_flags[4] != 0;

    // LDS carve-up (floats)
    const int XS = 36;          // row stride of X tile (conflict-free 16-byte reads)
    const int XTS = R + 4;      // row stride of X^T tile
    float *Xs = lds;                        // [R][36]
    float *XTs = Xs + R * XS;               // [32][R+4]
    float *Ys = XTs + 32 * XTS;             // [R]
    float *Ypart = Ys + R;                  // [WU][R]  partial Ypred per unit-wave
    float *Gs = Ypart + WU * R;             // [R]      dZ2 per row
    float *Rs2 = Gs + R;                    // [R]      squared residual per row
    float *Pred = Rs2 + R;                  // [WR][32][U+1] per-row-wave partial P
    const int PS = U + 1;                   // Pred row stride (conflict-free column reads)
    float *Wown = Pred + WR * 32 * PS;      // [upw][33] owned units (master copy)
    float *Sse = Wown + p.upw * 33;         // [8]

    if (active && !aborted) {
        // ---- initial weights --------------------------------------------------
        const int upw = p.upw;
        // B operand of Z1 for my unit tiles: W1[8*lq + t][u0 + li]
        float w1b[NUW][8];
        float w2v[NUW];
#pragma unroll
        for (int u = 0; u < NUW; ++u) {
            const int ul = (wu + u * WU) * 16 + li;              // unit index inside group
            const int ug = gx * U + ul;                          // global unit index
#pragma unroll
            for (int t = 0; t < 8; ++t) w1b[u][t] = a.W1[(8 * lq + t) * a.hidden + ug];
            w2v[u] = a.W2[ug];
        }
        for (int i = tid; i < upw * 33; i += 256) {
            const int jl = i / 33, k = i % 33;
            const int ug = gx * U + gb * upw + jl;
            Wown[i] = k < 32 ? a.W1[k * a.hidden + ug] : a.W2[ug];
        }
        double epoch_sse = 0.0;
        __syncthreads();

        const int64_t spe = (a.n + a.batch - 1) / a.batch;
        for (int64_t s = 0; s < a.steps; ++s) {
            const uint32_t tag = a.tag_base + (uint32_t)s;
            const int par = (int)(s & 1);
            const int64_t e = s / spe, sb = s % spe;
            const int64_t off = sb * a.batch;
            const int64_t nb = (a.n - off < a.batch) ? a.n - off : a.batch;
            const int64_t row0 = (int64_t)gb * R;
            const int rc = (int)(nb - row0 <= 0 ? 0 : (nb - row0 < R ? nb - row0 : R));
            const float scale = 2.0f / (float)nb;
            sync.deadline = now_ticks() + a.timeout_ticks;

            // ---- 1. stage rows: X tile, X^T tile, Y ---------------------------
            {
                const int32_t *order = a.perm ? a.perm + e * a.n : nullptr;   // epoch order
                const int64_t base = off + row0;                                // position in it
                for (int i = tid; i < R * 8; i += 256) {
                    const int r = i >> 3, c4 = (i & 7) * 4;
                    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                    if (r < rc) {
                        const int64_t row = gather_row(order, base + r, a.n_rows, a.err);
                        v = *reinterpret_cast<const float4 *>(a.X + row * D_IN + c4);
                    }
                    *reinterpret_cast<float4 *>(Xs + r * XS + c4) = v;
                    XTs[(c4 + 0) * XTS + r] = v.x;
                    XTs[(c4 + 1) * XTS + r] = v.y;
                    XTs[(c4 + 2) * XTS + r] = v.z;
                    XTs[(c4 + 3) * XTS + r] = v.w;
                }
                for (int r = tid; r < R; r += 256) {
                    float y = 0.f;
                    if (r < rc) y = a.Y[gather_row(order, base + r, a.n_rows, a.err)];
                    Ys[r] = y;
                }
            }
            __syncthreads();

            // ---- 2. forward: Z1 tiles, mask bits, partial Ypred --------------------
            uint32_t mbits = 0;   // bit (rt*NUW + u)*4 + v
#pragma unroll
            for (int rt = 0; rt < RTW; ++rt) {
                const int rtile = wr + rt * WR;
                if (rtile * 16 < R) {
                    const float *xr = Xs + (rtile * 16 + li) * XS + 8 * lq;
                    const float4 xa = *reinterpret_cast<const float4 *>(xr);
                    const float4 xb = *reinterpret_cast<const float4 *>(xr + 4);
                    const float xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
                    float yp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int u = 0; u < NUW; ++u) {
                        f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int t = 0; t < 8; ++t)
                            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[t], w1b[u][t], acc, 0, 0, 0);
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const float z = acc[v];
                            const bool on = z > 0.0f;                       // ReLU'(z) = [z > 0]
                            mbits |= (on ? 1u : 0u) << ((rt * NUW + u) * 4 + v);
                            yp[v] = fmaf(on ? z : 0.0f, w2v[u], yp[v]);     // eqs. 12-13
                        }
                    }
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float sv = sum16(yp[v]);
                        if (li == 0) Ypart[wu * R + rtile * 16 + 4 * lq + v] = sv;
                    }
                }
            }
            __syncthreads();

            // ---- 3. exchange A: partial Ypred across groups ------------------------
            // row sums over unit waves (fixed order), then over groups (fixed order);
            // thread r owns row r from here to the residual
            for (int r = tid; r < R; r += 256) {
                float v = 0.f;
                for (int w = 0; w < WU; ++w) v += Ypart[w * R + r];
                Gs[r] = v;
            }
            if (PX > 1) {
                uint64_t *xa = a.xch + ((size_t)(par * PR + gb) * PX) * p.rmax;
                for (int r = tid; r < R; r += 256) st_dev(xa + (size_t)gx * p.rmax + r, pack(Gs[r], tag));
                if (tid < PX) (void)wait_word(xa + (size_t)tid * p.rmax, tag, sync, aborted);
                __syncthreads();
                for (int r = tid; r < R; r += 256) {
                    float v = 0.f;
                    for (int x = 0; x < PX; ++x) v += wait_word(xa + (size_t)x * p.rmax + r, tag, sync, aborted);
                    Gs[r] = v;
                }
            }
            // residual, squared residual, dZ2 (eqs. 14-15)
            for (int r = tid; r < R; r += 256) {
                float gv = 0.f, r2 = 0.f;
                if (r < rc) {
                    const float res = Gs[r] - Ys[r];
                    r2 = res * res;
                    gv = scale * res;
                }
                Gs[r] = gv;
                Rs2[r] = r2;
            }
            __syncthreads();
            if (wave == 0) {      // batch SSE of my rows, fixed order
                float t = 0.f;
                for (int r = lane; r < R; r += 64) t += Rs2[r];
                t = sum32(t);
                t += __shfl_xor(t, 32, 64);
                if (lane == 0) Sse[0] = t;
            }

            // ---- 4. backward: P = X^T (dZ2 (.) mask) --------------------------------
            f4 pacc[2][NUW];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int u = 0; u < NUW; ++u) pacc[kt][u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int rt = 0; rt < RTW; ++rt) {
                const int rtile = wr + rt * WR;
                if (rtile * 16 < R) {
                    const int rb = rtile * 16 + 4 * lq;
                    const float4 g4 = *reinterpret_cast<const float4 *>(Gs + rb);
                    const float gv[4] = {g4.x, g4.y, g4.z, g4.w};
                    float xt[2][4];
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) {
                        const float4 t4 = *reinterpret_cast<const float4 *>(XTs + (kt * 16 + li) * XTS + rb);
                        xt[kt][0] = t4.x; xt[kt][1] = t4.y; xt[kt][2] = t4.z; xt[kt][3] = t4.w;
                    }
#pragma unroll
                    for (int u = 0; u < NUW; ++u) {
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const bool on = (mbits >> ((rt * NUW + u) * 4 + v)) & 1u;
                            const float gmv = on ? gv[v] : 0.0f;     // dZ2 (.) ReLU'(Z1)
#pragma unroll
                            for (int kt = 0; kt < 2; ++kt)
                                pacc[kt][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xt[kt][v], gmv, pacc[kt][u], 0, 0, 0);
                        }
                    }
                }
            }
            // per-row-wave partial P to LDS: Pred[wr][k][ul]
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int u = 0; u < NUW; ++u) {
                    const int ul = (wu + u * WU) * 16 + li;
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        Pred[(wr * 32 + kt * 16 + 4 * lq + v) * PS + ul] = pacc[kt][u][v];
                }
            __syncthreads();

            // ---- 5. exchange B: reduce-scatter of P inside the group ---------------
            {
                // workgroup partial (row waves summed in order) -> tagged words
                uint64_t *rsw = a.rs + ((size_t)(par * PX + gx) * PR + gb) * p.rs_stride;
                for (int i = tid; i < 32 * U; i += 256) {
                    const int ul = i / 32, k = i % 32;
                    float v = 0.f;
                    for (int w = 0; w < WR; ++w) v += Pred[(w * 32 + k) * PS + ul];
                    st_loc(rsw + (size_t)ul * 32 + k, pack(v, tag), plain);
                }
                if (tid == 0) st_loc(rsw + (size_t)U * 32, pack(gx == 0 ? Sse[0] : 0.f, tag), plain);
                // poll the last word of every peer, then reduce my units
                const uint64_t *rsg = a.rs + ((size_t)(par * PX + gx) * PR) * p.rs_stride;
                if (tid < PR) (void)wait_word(rsg + (size_t)tid * p.rs_stride + (size_t)U * 32, tag, sync, aborted);
                __syncthreads();
                for (int i = tid; i < upw * 32; i += 256) {
                    const int jl = i / 32, k = i % 32;
                    const int ul = gb * upw + jl;
                    float v = 0.f;
                    for (int b2 = 0; b2 < PR; ++b2)
                        v += wait_word(rsg + (size_t)b2 * p.rs_stride + (size_t)ul * 32 + k, tag, sync, aborted);
                    Pred[jl * 32 + k] = v;      // P[k][unit] of my owned units (reuse LDS)
                }
                if (tid == 0 && gx == 0 && gb == 0) {
                    float v = 0.f;
                    for (int b2 = 0; b2 < PR; ++b2)
                        v += wait_word(rsg + (size_t)b2 * p.rs_stride + (size_t)U * 32, tag, sync, aborted);
                    Sse[1] = v;
                }
                __syncthreads();
            }

            // ---- update my units (eq. 19) or emit gradients -------------------------
            // thread (jl, k): k = tid % 32 inside a 32-lane half wave
            for (int i = tid; i < upw * 32; i += 256) {
                const int jl = i / 32, k = i % 32;
                const float pk = Pred[jl * 32 + k];
                const float w1 = Wown[jl * 33 + k];
                const float w2 = Wown[jl * 33 + 32];
                const float dw2 = sum32(w1 * pk);              // dW2_j = sum_k W1_kj P_kj
                const float dw1 = w2 * pk;                      // dW1_kj = W2_j P_kj
                const int ug = gx * U + gb * upw + jl;
                if (a.mode == 1) {
                    a.dW1[k * a.hidden + ug] = dw1;
                    if (k == 0) a.dW2[ug] = dw2;
                } else {
                    Wown[jl * 33 + k] = w1 - a.lr * dw1;
                    if (k == 0) Wown[jl * 33 + 32] = w2 - a.lr * dw2;
                }
            }
            if (tid == 0 && gx == 0 && gb == 0) {
                const float L = Sse[1] / (float)nb;               // eq. 14
                if (a.loss) a.loss[0] = L;
                if (a.step_loss) a.step_loss[s] = L;
                if (sb == 0) epoch_sse = 0.0;
                epoch_sse += (double)Sse[1];
                if (a.epoch_loss) a.epoch_loss[e] = (float)(epoch_sse * (double)a.inv_n);
            }
            if (a.mode == 1) break;   // gradient only: one step, weights untouched
            __syncthreads();

            // ---- 6. exchange C: all-gather the group's updated slice ----------------
            {
                uint64_t *agg = a.ag + ((size_t)(par * PX + gx)) * (size_t)U * 33;
                for (int i = tid; i < upw * 33; i += 256) {
                    const int jl = i / 33, k = i % 33;
                    st_loc(agg + (size_t)(gb * upw + jl) * 33 + k, pack(Wown[i], tag), plain);
                }
                // poll the first word of each owner, then read my B-operand slice
                if (tid < PR) (void)wait_word(agg + (size_t)(tid * upw) * 33, tag, sync, aborted);
                __syncthreads();
#pragma unroll
                for (int u = 0; u < NUW; ++u) {
                    const int ul = (wu + u * WU) * 16 + li;
#pragma unroll
                    for (int t = 0; t < 8; ++t) w1b[u][t] = wait_word(agg + (size_t)ul * 33 + 8 * lq + t, tag, sync, aborted);
                    w2v[u] = wait_word(agg + (size_t)ul * 33 + 32, tag, sync, aborted);
                }
            }
            if (__syncthreads_or(aborted ? 1 : 0)) break;
        }

        // ---- final weights in the caller's layout ---------------------------------
        __syncthreads();
        if (a.mode == 0 && tid == 0 && gx == 0 && gb == 0 && a.epoch_loss) {
            const int64_t last_epoch = a.steps > 0 ? (a.steps - 1) / spe : -1;
            for (int64_t e2 = last_epoch + 1; e2 < a.epochs; ++e2) a.epoch_loss[e2] = 0.0f;
        }
        if (a.mode == 0) {
            for (int i = tid; i < upw * 33; i += 256) {
                const int jl = i / 33, k = i % 33;
                const int ug = gx * U + gb * upw + jl;
                if (k < 32) a.W1[k * a.hidden + ug] = Wown[i];
                else a.W2[ug] = Wown[i];
            }
        }
    }

    // ---- teardown: the last workgroup out clears the registration counters ------
    __syncthreads();
    if (tid == 0) {
        const int done = __hip_atomic_fetch_add(&a.reg[10], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if (done == (int)gridDim.x - 1) {
            for (int i = 0; i < 16; ++i)
                __hip_atomic_store(&a.reg[i], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.abort, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ---------------------------------------------------------------------------
// Host side: plan and launch
// ---------------------------------------------------------------------------

static int pow2_floor(int64_t v) {
    int p = 1;
    while ((int64_t)p * 2 <= v) p *= 2;
    return p;
}

static bool valid_tile(int nuw, int rtw) {
    return (nuw == 1 || nuw == 2 || nuw == 4 || nuw == 8) &&
           (rtw == 1 || rtw == 2 || rtw == 4 || rtw == 8) && nuw * rtw <= 8;
}

// Fill a plan for PX groups; false when the shape does not fit the kernel.
static bool plan_for(int hidden, int64_t batch, int px, TrainPlan *pl) {
    if (hidden % px) return false;
    const int U = hidden / px;
    if (U < 16 || U % 16) return false;
    int64_t want = (batch + 15) / 16;                 // at least 16 rows per workgroup
    int pr = pow2_floor(want < 1 ? 1 : want);
    if (pr > 32) pr = 32;
    if (pr > U) pr = pow2_floor(U);
    int64_t R = (batch + pr - 1) / pr;
    R = (R + 15) / 16 * 16;
    if (R > RMAX) return false;
    const int NR = (int)(R / 16), NU = U / 16;
    const int wr = NR >= 4 ? 4 : (NR >= 2 ? 2 : 1);
    const int wu = 4 / wr;
    if (NU % wu) return false;
    const int nuw = NU / wu, rtw = (NR + wr - 1) / wr;
    if (!valid_tile(nuw, rtw)) return false;
    pl->px = px;
    pl->pr = pr;
    pl->R = (int)R;
    pl->U = U;
    pl->wr = wr;
    pl->wu = wu;
    pl->nuw = nuw;
    pl->rtw = rtw;
    pl->upw = U / pr;
    pl->rmax = RMAX;
    pl->rs_stride = (U * 32 + 1 + 31) / 32 * 32;
    pl->grid = 8 * pr;
    const size_t floats = (size_t)R * 36 + 32 * (size_t)(R + 4) + (size_t)R * (4 + wu) +
                          (size_t)wr * 32 * (U + 1) + (size_t)pl->upw * 33 + 8;
    size_t bytes = floats * sizeof(float);
    const size_t one_per_cu = 84 * 1024;   // > half of the 160 KB LDS: one workgroup per CU
    pl->lds = bytes > one_per_cu ? bytes : one_per_cu;
    return pl->lds <= 160 * 1024;
}

// Modelled step time: MFMA work of one wave plus the exchange latencies
// measured on MI355X (about 1.2 us across XCDs, 0.5 us inside one).
static double plan_cost(const TrainPlan &pl) {
    const double mfma_cycles = 32.0 * 16.0 * pl.nuw * pl.rtw;
    const double compute = 1.5 * mfma_cycles / 2.4e9;
    return compute + (pl.px > 1 ? 1.2e-6 : 0.0) + 1.0e-6;
}

bool plan_train(int hidden, int64_t batch, TrainPlan *plan) {
    const char *force = getenv("MLP_PX");
    const int fpx = force ? atoi(force) : 0;
    bool found = false;
    TrainPlan best;
    double best_cost = 0.0;
    for (int px : {1, 2, 4, 8}) {
        if (fpx && px != fpx) continue;
        TrainPlan pl;
        if (!plan_for(hidden, batch, px, &pl)) continue;
        const double cst = plan_cost(pl);
        if (!found || cst < best_cost) {
            best = pl;
            best_cost = cst;
            found = true;
        }
    }
    if (found) *plan = best;
    return found;
}

size_t persist_words_xch() { return (size_t)2 * 32 * 8 * RMAX; }
size_t persist_words_rs(int hidden) { return (size_t)2 * 32 * ((size_t)hidden * 32 + 8 * 32); }
size_t persist_words_ag(int hidden) { return (size_t)2 * hidden * 33; }

template <int NUW, int RTW>
static hipError_t launch_t(Ctx &c, TrainArgs &a) {
    void *args[] = {&a};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&k_train<NUW, RTW>),
                                      dim3(a.plan.grid), dim3(256), args, (unsigned)a.plan.lds,
                                      c.stream);
}

hipError_t launch_train(Ctx &c, TrainArgs &a) {
    a.xch = c.xch;
    a.rs = c.rs;
    a.ag = c.ag;
    a.reg = c.ctl->reg;
    a.abort = &c.ctl->abort;
    a.err = &c.ctl->err;
    a.tag_base = c.tag_base;
    a.timeout_ticks = 200000000ull;   // 2 s
    const char *fc = getenv("MLP_FORCE_COHERENT");
    a.force_coherent = (fc && fc[0] == '1') ? 1 : 0;
    // tags of the next call start past every tag this call can use
    c.tag_base += (uint32_t)(a.steps + 2);
    if (c.tag_base < 1) c.tag_base = 1;
    const int nuw = a.plan.nuw, rtw = a.plan.rtw;
#define MLP_TRY(NU, RT) \
    if (nuw == NU && rtw == RT) return launch_t<NU, RT>(c, a);
    MLP_TRY(1, 1) MLP_TRY(1, 2) MLP_TRY(1, 4) MLP_TRY(1, 8)
    MLP_TRY(2, 1) MLP_TRY(2, 2) MLP_TRY(2, 4)
    MLP_TRY(4, 1) MLP_TRY(4, 2)
    MLP_TRY(8, 1)
#undef MLP_TRY
    return hipErrorInvalidValue;
}

}  // namespace mlp
