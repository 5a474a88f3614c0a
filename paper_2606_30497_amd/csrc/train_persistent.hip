// train_persistent.hip -- single-launch fused mini-batch SGD trainer for the
// d-h-1 ReLU/MSE network (paper Sec. III eqs. 11-19, d = 32), for gfx950.
//
// Decomposition (one workgroup per CU, 4 waves each):
//   - the hidden units are split over PX groups of workgroups; each group lives
//     on one XCD (8 XCDs, one L2 each) and owns U = h/PX units;
//   - inside a group, PR workgroups split the rows of every mini-batch (R rows
//     each) and keep the group's W1 slice [32 x U] and W2 slice [U] in registers.
// One SGD step is then:
//   1. stage the step's rows (gathered through the epoch permutation one step
//      earlier by the loader waves) in LDS, as X [R x 32] and X^T [32 x R];
//   2. Z1 = X W1 on fp32 MFMA (16x16x4); ReLU mask bits and the partial Ypred
//      over the group's units stay in registers (eqs. 11-13);
//   3. exchange A (across XCDs, PX-way): sum the PX partial Ypred of each row in
//      group order -> full Ypred, residual, dZ2 = (2/n_b) r (eqs. 14-15);
//   4. P = X^T (dZ2 (.) [Z1 > 0]) on MFMA over the workgroup's rows; then
//      dW1 = P diag(W2) and dW2_j = sum_k W1_kj P_kj, which equal eqs. 16-18
//      (H_rj = [Z1_rj > 0] sum_k X_rk W1_kj);
//   5. exchange B (inside the XCD, PR-way reduce-scatter): workgroup b sums, in
//      workgroup order, the P columns of the units it owns and applies
//      W -= lr dW to them (eq. 19);
//   6. exchange C (inside the XCD, all-gather): every workgroup of the group
//      reads the updated slice.
// Exchanges use 64-bit words holding (fp32 value, 32-bit step tag). Writers
// never wait; a reader polls one word per peer, then loads the rest and retries
// any word whose tag is not yet current. Every sum runs in a fixed order, so
// results are bitwise reproducible and identical in every group that computes
// them. No floating-point atomics are used.
//
// Memory scopes: exchange A stores and all exchange loads are device-coherent
// (sc1). Exchanges B and C stay inside one XCD, whose L2 is shared: their
// stores are plain (write-through L1 into the XCD's L2) when every group was
// verified at start-up to sit on one XCD (hardware XCC id); otherwise they are
// device-coherent as well, which is correct for any placement.
//
// Every shape parameter is a compile-time constant of the instantiation
// (Shape<PX, PR, R, U>), so loops unroll and addressing folds to immediates.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

typedef float f4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Shapes
// ---------------------------------------------------------------------------

template <int PX_, int PR_, int R_, int U_>
struct Shape {
    static constexpr int PX = PX_, PR = PR_, R = R_, U = U_;
    static constexpr int H = PX * U;                       // hidden units
    static constexpr int NR = R / 16, NU = U / 16;         // row / unit tiles
    static constexpr int WR = NR >= 4 ? 4 : NR;            // waves along rows
    static constexpr int WU = 4 / WR;                      // waves along units
    static constexpr int NUW = NU / WU;                    // unit tiles per wave
    static constexpr int RTW = NR / WR;                    // row tiles per wave
    static constexpr int UPW = U / PR;                     // units owned per workgroup
    static constexpr int XS = 36;                          // X tile row stride
    static constexpr int XTS = R + 4;                      // X^T tile row stride
    static constexpr int PS = U + 1;                       // P partial row stride
    static constexpr int RSW = 32 * U;                     // B-exchange words (+1 sse)
    static constexpr int RS_STRIDE = (RSW + 1 + 31) / 32 * 32;
    static constexpr int RPT = R / 16;                     // rows per loader thread
    // LDS carve-up, in floats
    static constexpr int O_XS = 0;
    static constexpr int O_XT = O_XS + R * XS;
    static constexpr int O_Y = O_XT + 32 * XTS;
    static constexpr int O_YP = O_Y + R;
    static constexpr int O_G = O_YP + WU * R;
    static constexpr int O_R2 = O_G + R;
    static constexpr int O_P = O_R2 + R;
    static constexpr int O_WO = O_P + WR * 32 * PS;
    static constexpr int O_SSE = (O_WO + UPW * 33 + 3) / 4 * 4;
    static constexpr int O_WSL = O_SSE + 8;
    static constexpr int LDS_FLOATS = O_WSL + U * 33;

    static_assert(R % 16 == 0 && U % 16 == 0, "tiles");
    static_assert(WR * WU == 4 && NR % WR == 0 && NU % WU == 0, "wave split");
    static_assert(NUW >= 1 && RTW >= 1 && NUW * RTW <= 8, "mask bits");
    static_assert(U % PR == 0 && UPW >= 1, "ownership");
    static_assert(R <= RMAX && R <= 256, "rows");
    static_assert(PX >= 1 && PX <= 8 && PR >= 1 && PR <= 32, "grid");
};

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

struct Waiter {
    int32_t *abort;      // kernel-wide abort word (set on a timeout)
    int32_t *err;        // sticky error word
    uint64_t deadline;   // s_memrealtime ticks
    bool aborted;

    __device__ __forceinline__ void check() {
        if (__hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
            aborted = true;
        } else if (now_ticks() > deadline) {
            __hip_atomic_store(err, (int32_t)MLP_ERR_TIMEOUT_CODE, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            aborted = true;
        }
    }
    // spin until the word at p carries tag
    __device__ __forceinline__ void poll(const uint64_t *p, uint32_t tag) {
        uint32_t spins = 0;
        while (!aborted && tag_of(ld_dev(p)) != tag)
            if ((++spins & 255u) == 0) check();
    }
    // N words at p + i*stride: all loads issued first, stale words reloaded;
    // out[i] = value of word i. Every load is retired before returning.
    template <int N>
    __device__ __forceinline__ void load(const uint64_t *p, size_t stride, uint32_t tag,
                                         float (&out)[N]) {
        uint64_t w[N];
#pragma unroll
        for (int i = 0; i < N; ++i) w[i] = ld_dev(p + i * stride);
        uint32_t spins = 0;
        while (true) {
            bool ok = true;
#pragma unroll
            for (int i = 0; i < N; ++i) ok = ok && tag_of(w[i]) == tag;
            if (ok || aborted) break;
#pragma unroll
            for (int i = 0; i < N; ++i)
                if (tag_of(w[i]) != tag) w[i] = ld_dev(p + i * stride);
            if ((++spins & 63u) == 0) check();
        }
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): no load left in flight
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = val_of(w[i]);
    }
};

// Sum over each row of 16 lanes by DPP right shifts (bound_ctrl: lanes shifted
// in from outside the row read 0); lane 15 of the row holds the total, summed
// in a fixed order.
__device__ __forceinline__ float row16_sum(float v) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x111, 0xF, 0xF, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x112, 0xF, 0xF, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x114, 0xF, 0xF, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x118, 0xF, 0xF, true));
    return v;
}
// Butterfly sum over aligned groups of 32 lanes (every lane gets the total).
__device__ __forceinline__ float sum32(float v) {
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 1, 64);
    return v;
}

// Optional phase timestamps (s_memrealtime, 100 MHz): workgroup (0, 0) for the
// first TRACE_STEPS steps, or every workgroup for steps [16, 24).
constexpr int TRACE_STEPS = 48;
constexpr int TRACE_ALL_FIRST = 16, TRACE_ALL_STEPS = 8;
#define TRACE(ph)                                                                          \
    do {                                                                                   \
        if (a.trace && tid == 0 && gx == 0 && gb == 0 && s < TRACE_STEPS)                  \
            a.trace[s * 8 + (ph)] = now_ticks();                                           \
        if (a.trace_all && tid == 0 && s >= TRACE_ALL_FIRST &&                             \
            s < TRACE_ALL_FIRST + TRACE_ALL_STEPS)                                         \
            a.trace_all[((gx * S::PR + gb) * TRACE_ALL_STEPS + (s - TRACE_ALL_FIRST)) * 8 + \
                        (ph)] = now_ticks();                                               \
    } while (0)

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
// Waves: wave w takes row tiles {w % WR + i*WR} and unit tiles {w / WR + i*WU}.
// Waves 2 and 3 also gather the next step's rows ("loader" waves); waves 0 and
// 1 own the rows in exchange A and the residual.
template <class S>
__global__ __launch_bounds__(256) void k_train(const TrainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int s_flags[8];   // 0: group x, 1: rank b, 2: plain local stores, 3: abort, 4: active

    constexpr int R = S::R, U = S::U, PR = S::PR, PX = S::PX, H = S::H;
    constexpr int WR = S::WR, WU = S::WU, NUW = S::NUW, RTW = S::RTW, UPW = S::UPW;
    constexpr int XS = S::XS, XTS = S::XTS, PS = S::PS;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lq = lane >> 4, li = lane & 15;   // lane group (0..3) and index in group
    const int wr = wave % WR, wu = wave / WR;

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
        int gx_, gb_, active;
        if (placed) {
            gx_ = (int)x_hw;
            gb_ = rank_x;
            active = gx_ < PX && gb_ < PR;
        } else {
            gx_ = rank_g / PR;
            gb_ = rank_g % PR;
            active = rank_g < PX * PR;
        }
        s_flags[0] = gx_;
        s_flags[1] = gb_;
        s_flags[2] = placed ? 1 : 0;
        s_flags[3] = ab;
        s_flags[4] = active;
    }
    __syncthreads();
    const int gx = s_flags[0], gb = s_flags[1];
    const bool plain = s_flags[2] != 0;
    const bool active = s_flags[4] != 0;
    Waiter wt{a.abort, a.err, 0, s_flags[3] != 0};

    float *Xs = lds + S::O_XS;     // [R][36]
    float *XTs = lds + S::O_XT;    // [32][R+4]
    float *Ys = lds + S::O_Y;      // [R]
    float *Ypart = lds + S::O_YP;  // [WU][R]  partial Ypred per unit-wave
    float *Gs = lds + S::O_G;      // [R]      Ypred, then dZ2, per row
    float *Rs2 = lds + S::O_R2;    // [R]      squared residual per row
    float *Pred = lds + S::O_P;    // [WR][32][U+1] per-row-wave partial P
    float *Wown = lds + S::O_WO;   // [UPW][33] owned units (master copy)
    float *Sse = lds + S::O_SSE;   // [8]
    float *Wsl = lds + S::O_WSL;   // [U][33]  the group's slice after exchange C

    if (active && !wt.aborted) {
        // ---- initial weights --------------------------------------------------
        float w1b[NUW][8];   // B operand of Z1: W1[8*lq + t][unit (wu + u*WU)*16 + li]
        float w2v[NUW];
#pragma unroll
        for (int u = 0; u < NUW; ++u) {
            const int ug = gx * U + (wu + u * WU) * 16 + li;
#pragma unroll
            for (int t = 0; t < 8; ++t) w1b[u][t] = a.W1[(8 * lq + t) * H + ug];
            w2v[u] = a.W2[ug];
        }
        for (int i = tid; i < UPW * 33; i += 256) {
            const int jl = i / 33, k = i % 33;
            const int ug = gx * U + gb * UPW + jl;
            Wown[i] = k < 32 ? a.W1[k * H + ug] : a.W2[ug];
        }
        double epoch_sse = 0.0;
        // retire the initial loads before the step loop (see the row pipeline)
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();

        // ---- row pipeline (loader waves 2 and 3) --------------------------------
        // Epoch-order indices are loaded two steps ahead and X/Y rows one step
        // ahead, into registers that are read only when the next step stages its
        // rows; the loader waves issue them right after exchange A, so they land
        // during the rest of the step.
        const int64_t spe = (a.n + a.batch - 1) / a.batch;
        const int64_t row0 = (int64_t)gb * R;
        const bool loader = tid >= 128;
        const int lt = tid - 128, lc4 = (lt & 7) * 4, lr = lt >> 3;   // 16 rows per pass
        int32_t pidx[S::RPT];
        float4 pfx[S::RPT];
        float pfy[S::RPT];
        // issue the index loads of the step at (epoch e, offset off): raw values
        auto fetch_idx = [&](int64_t e, int64_t off) {
            if (!a.perm) return;
            const int32_t *order = a.perm + e * a.n;
#pragma unroll
            for (int j = 0; j < S::RPT; ++j) {
                int64_t pos = off + row0 + lr + 16 * j;
                pos = pos < a.n ? pos : a.n - 1;            // always a valid address
                pidx[j] = order[pos];
            }
        };
        // issue the X/Y loads of the step at offset off from indices fetched earlier
        auto fetch_rows = [&](int64_t off) {
            const int64_t nb = a.n - off < a.batch ? a.n - off : a.batch;
            const int64_t rcl = nb - row0;
#pragma unroll
            for (int j = 0; j < S::RPT; ++j) {
                const int r = lr + 16 * j;
                float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                float y = 0.f;
                if (r < rcl) {
                    int64_t row = a.perm ? (int64_t)pidx[j] : off + row0 + r;
                    if (row < 0 || row >= a.n_rows) {
                        __hip_atomic_store(a.err, (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                        row = 0;
                    }
                    v = *reinterpret_cast<const float4 *>(a.X + row * D_IN + lc4);
                    if (lc4 == 0) y = a.Y[row];
                }
                pfx[j] = v;
                pfy[j] = y;
            }
        };
        // step bookkeeping: (epoch, step in epoch) of steps s, s+1 and s+2
        int64_t e0 = 0, sb0 = 0;
        int64_t e1 = 0, sb1 = 1;
        if (sb1 == spe) { sb1 = 0; ++e1; }
        int64_t e2 = e1, sb2 = sb1 + 1;
        if (sb2 == spe) { sb2 = 0; ++e2; }
        if (loader) {
            if (a.steps > 0) {
                fetch_idx(0, 0);
                fetch_rows(0);
            }
            if (a.steps > 1) fetch_idx(e1, sb1 * a.batch);
        }

        for (int64_t s = 0; s < a.steps; ++s) {
            const uint32_t tag = a.tag_base + (uint32_t)s;
            const int par = (int)(s & 1);
            const int64_t off = sb0 * a.batch;
            const int64_t nb = (a.n - off < a.batch) ? a.n - off : a.batch;
            const int rc = (int)(nb - row0 <= 0 ? 0 : (nb - row0 < R ? nb - row0 : R));
            const float scale = 2.0f / (float)nb;
            wt.deadline = now_ticks() + a.timeout_ticks;
            TRACE(0);

            // ---- 1. stage the rows gathered during the previous step --------------
            if (loader) {
#pragma unroll
                for (int j = 0; j < S::RPT; ++j) {
                    const int r = lr + 16 * j;
                    const float4 v = pfx[j];
                    *reinterpret_cast<float4 *>(Xs + r * XS + lc4) = v;
                    XTs[(lc4 + 0) * XTS + r] = v.x;
                    XTs[(lc4 + 1) * XTS + r] = v.y;
                    XTs[(lc4 + 2) * XTS + r] = v.z;
                    XTs[(lc4 + 3) * XTS + r] = v.w;
                    if (lc4 == 0) Ys[r] = pfy[j];
                }
            }
            __syncthreads();

            // ---- 2. forward: Z1 tiles, mask bits, partial Ypred --------------------
            uint32_t mbits = 0;   // bit (rt*NUW + u)*4 + v
#pragma unroll
            for (int rt = 0; rt < RTW; ++rt) {
                const int rtile = wr + rt * WR;
                const float *xr = Xs + (rtile * 16 + li) * XS + 8 * lq;
                const float4 xa = *reinterpret_cast<const float4 *>(xr);
                const float4 xb = *reinterpret_cast<const float4 *>(xr + 4);
                const float xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
                float yp[4] = {0.f, 0.f, 0.f, 0.f};
                f4 acc[NUW];
#pragma unroll
                for (int u = 0; u < NUW; ++u) acc[u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < 8; ++t)
#pragma unroll
                    for (int u = 0; u < NUW; ++u)
                        acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[t], w1b[u][t], acc[u], 0, 0, 0);
#pragma unroll
                for (int u = 0; u < NUW; ++u)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float z = acc[u][v];
                        const bool on = z > 0.0f;                       // ReLU'(z) = [z > 0]
                        mbits |= (on ? 1u : 0u) << ((rt * NUW + u) * 4 + v);
                        yp[v] = fmaf(on ? z : 0.0f, w2v[u], yp[v]);     // eqs. 12-13
                    }
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float sv = row16_sum(yp[v]);
                    if (li == 15) Ypart[wu * R + rtile * 16 + 4 * lq + v] = sv;
                }
            }
            __syncthreads();
            TRACE(1);

            // ---- 3. exchange A: partial Ypred across groups ------------------------
            // thread r % 128 (waves 0-1) owns row r through the residual
            if (tid < 128) {
#pragma unroll
                for (int r0 = 0; r0 < R; r0 += 128) {
                    const int r = r0 + tid;
                    if (r < R) {
                        float v = 0.f;
#pragma unroll
                        for (int w = 0; w < WU; ++w) v += Ypart[w * R + r];
                        Gs[r] = v;
                    }
                }
            }
            if constexpr (PX > 1) {
                uint64_t *xa = a.xch + (size_t)((par * PR + gb) * PX) * RMAX;
                if (tid < 128) {
#pragma unroll
                    for (int r0 = 0; r0 < R; r0 += 128) {
                        const int r = r0 + tid;
                        if (r < R) st_dev(xa + gx * RMAX + r, pack(Gs[r], tag));
                    }
                }
                if (tid < PX) wt.poll(xa + tid * RMAX, tag);
                __syncthreads();
                if (tid < 128) {
#pragma unroll
                    for (int r0 = 0; r0 < R; r0 += 128) {
                        const int r = r0 + tid;
                        if (r < R) {
                            float vals[PX];
                            wt.load<PX>(xa + r, RMAX, tag, vals);
                            float v = 0.f;
#pragma unroll
                            for (int x = 0; x < PX; ++x) v += vals[x];
                            Gs[r] = v;
                        }
                    }
                }
            }
            TRACE(2);
            // gather the next step's rows (see the row pipeline above)
            if (loader) {
                if (s + 1 < a.steps) fetch_rows(sb1 * a.batch);
                if (s + 2 < a.steps) fetch_idx(e2, sb2 * a.batch);
            }
            // residual, squared residual, dZ2 (eqs. 14-15)
            if (tid < 128) {
#pragma unroll
                for (int r0 = 0; r0 < R; r0 += 128) {
                    const int r = r0 + tid;
                    if (r < R) {
                        float gv = 0.f, r2 = 0.f;
                        if (r < rc) {
                            const float res = Gs[r] - Ys[r];
                            r2 = res * res;
                            gv = scale * res;
                        }
                        Gs[r] = gv;
                        Rs2[r] = r2;
                    }
                }
            }
            __syncthreads();
            if (wave == 0) {      // SSE of my rows, fixed order
                float t = 0.f;
#pragma unroll
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
                const int rb = (wr + rt * WR) * 16 + 4 * lq;
                const float4 g4 = *reinterpret_cast<const float4 *>(Gs + rb);
                const float gv[4] = {g4.x, g4.y, g4.z, g4.w};
                float xt[2][4];
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const float4 t4 = *reinterpret_cast<const float4 *>(XTs + (kt * 16 + li) * XTS + rb);
                    xt[kt][0] = t4.x; xt[kt][1] = t4.y; xt[kt][2] = t4.z; xt[kt][3] = t4.w;
                }
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int u = 0; u < NUW; ++u) {
                        const bool on = (mbits >> ((rt * NUW + u) * 4 + v)) & 1u;
                        const float gmv = on ? gv[v] : 0.0f;     // dZ2 (.) ReLU'(Z1)
#pragma unroll
                        for (int kt = 0; kt < 2; ++kt)
                            pacc[kt][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xt[kt][v], gmv, pacc[kt][u], 0, 0, 0);
                    }
            }
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
            TRACE(3);

            // ---- 5. exchange B: reduce-scatter of P inside the group ---------------
            {
                uint64_t *rsg = a.rs + (size_t)((par * PX + gx) * PR) * S::RS_STRIDE;
                uint64_t *rsw = rsg + gb * S::RS_STRIDE;
                // my partial, row waves summed in order: word ul*32 + k
#pragma unroll
                for (int i0 = 0; i0 < S::RSW; i0 += 256) {
                    const int i = i0 + tid;
                    const int ul = i >> 5, k = i & 31;
                    float v = 0.f;
#pragma unroll
                    for (int w = 0; w < WR; ++w) v += Pred[(w * 32 + k) * PS + ul];
                    st_loc(rsw + i, pack(v, tag), plain);
                }
                if (tid == 0) st_loc(rsw + S::RSW, pack(gx == 0 ? Sse[0] : 0.f, tag), plain);
                if (tid < PR) wt.poll(rsg + tid * S::RS_STRIDE + S::RSW, tag);
                __syncthreads();
                // the units I own: P[k][gb*UPW + jl], summed over workgroups in order
#pragma unroll
                for (int i0 = 0; i0 < UPW * 32; i0 += 256) {
                    const int i = i0 + tid;
                    if (i < UPW * 32) {
                        float vals[PR];
                        wt.load<PR>(rsg + gb * UPW * 32 + i, S::RS_STRIDE, tag, vals);
                        float v = 0.f;
#pragma unroll
                        for (int b2 = 0; b2 < PR; ++b2) v += vals[b2];
                        Pred[i] = v;
                    }
                }
                if (tid == 0 && gx == 0 && gb == 0) {
                    float vals[PR];
                    wt.load<PR>(rsg + S::RSW, S::RS_STRIDE, tag, vals);
                    float v = 0.f;
#pragma unroll
                    for (int b2 = 0; b2 < PR; ++b2) v += vals[b2];
                    Sse[1] = v;
                }
                __syncthreads();
            }
            TRACE(4);

            // ---- update my units (eq. 19) or emit gradients -------------------------
#pragma unroll
            for (int i0 = 0; i0 < UPW * 32; i0 += 256) {
                const int i = i0 + tid;
                if (i < UPW * 32) {
                    const int jl = i >> 5, k = i & 31;
                    const float pk = Pred[i];
                    const float w1 = Wown[jl * 33 + k];
                    const float w2 = Wown[jl * 33 + 32];
                    const float dw2 = sum32(w1 * pk);              // dW2_j = sum_k W1_kj P_kj
                    const float dw1 = w2 * pk;                      // dW1_kj = W2_j P_kj
                    const int ug = gx * U + gb * UPW + jl;
                    if (a.mode == 1) {
                        a.dW1[k * H + ug] = dw1;
                        if (k == 0) a.dW2[ug] = dw2;
                    } else {
                        Wown[jl * 33 + k] = w1 - a.lr * dw1;
                        if (k == 0) Wown[jl * 33 + 32] = w2 - a.lr * dw2;
                    }
                }
            }
            if (tid == 0 && gx == 0 && gb == 0) {
                const float L = Sse[1] / (float)nb;               // eq. 14
                if (a.loss) a.loss[0] = L;
                if (a.step_loss) a.step_loss[s] = L;
                if (sb0 == 0) epoch_sse = 0.0;
                epoch_sse += (double)Sse[1];
                if (a.epoch_loss) a.epoch_loss[e0] = (float)(epoch_sse * (double)a.inv_n);
            }
            if (a.mode == 1) break;   // gradient only: one step, weights untouched
            __syncthreads();
            TRACE(5);

            // ---- 6. exchange C: all-gather the group's updated slice ----------------
            {
                uint64_t *agg = a.ag + (size_t)((par * PX + gx) * U) * 33;
                for (int i = tid; i < UPW * 33; i += 256)
                    st_loc(agg + gb * UPW * 33 + i, pack(Wown[i], tag), plain);
                if (tid < PR) wt.poll(agg + tid * UPW * 33, tag);
                __syncthreads();
                constexpr int NW = U * 33, FULL = NW / 256, REST = NW % 256;
                if constexpr (FULL > 0) {
                    float vals[FULL];
                    wt.load<FULL>(agg + tid, 256, tag, vals);
#pragma unroll
                    for (int q = 0; q < FULL; ++q) Wsl[tid + 256 * q] = vals[q];
                }
                if constexpr (REST > 0) {
                    if (tid < REST) {
                        float vals[1];
                        wt.load<1>(agg + 256 * FULL + tid, 0, tag, vals);
                        Wsl[256 * FULL + tid] = vals[0];
                    }
                }
                __syncthreads();
#pragma unroll
                for (int u = 0; u < NUW; ++u) {
                    const int ul = (wu + u * WU) * 16 + li;
#pragma unroll
                    for (int t = 0; t < 8; ++t) w1b[u][t] = Wsl[ul * 33 + 8 * lq + t];
                    w2v[u] = Wsl[ul * 33 + 32];
                }
            }
            TRACE(6);
            // advance the step bookkeeping
            e0 = e1; sb0 = sb1;
            e1 = e2; sb1 = sb2;
            if (++sb2 == spe) { sb2 = 0; ++e2; }
            if (__syncthreads_or(wt.aborted ? 1 : 0)) break;
        }

        // ---- final weights in the caller's layout, epochs never reached ----------
        __syncthreads();
        if (a.mode == 0) {
            for (int i = tid; i < UPW * 33; i += 256) {
                const int jl = i / 33, k = i % 33;
                const int ug = gx * U + gb * UPW + jl;
                if (k < 32) a.W1[k * H + ug] = Wown[i];
                else a.W2[ug] = Wown[i];
            }
            if (tid == 0 && gx == 0 && gb == 0 && a.epoch_loss) {
                const int64_t last_epoch = a.steps > 0 ? (a.steps - 1) / spe : -1;
                for (int64_t e = last_epoch + 1; e < a.epochs; ++e) a.epoch_loss[e] = 0.0f;
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
// Host side: instantiations, plan and launch
// ---------------------------------------------------------------------------

template <class S>
static hipError_t launch_shape(hipStream_t stream, TrainArgs &a) {
    void *args[] = {&a};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&k_train<S>),
                                      dim3(a.plan.grid), dim3(256), args, (unsigned)a.plan.lds,
                                      stream);
}

template <class S>
static TrainPlan plan_of(int inst) {
    TrainPlan p;
    p.inst = inst;
    p.px = S::PX;
    p.pr = S::PR;
    p.R = S::R;
    p.U = S::U;
    p.wr = S::WR;
    p.wu = S::WU;
    p.nuw = S::NUW;
    p.rtw = S::RTW;
    p.upw = S::UPW;
    p.rmax = RMAX;
    p.rs_stride = S::RS_STRIDE;
    p.grid = 8 * S::PR;
    const size_t bytes = sizeof(float) * (size_t)S::LDS_FLOATS;
    const size_t one_per_cu = 84 * 1024;   // > half of the 160 KB LDS: one workgroup per CU
    p.lds = bytes > one_per_cu ? bytes : one_per_cu;
    return p;
}

// The instantiated shapes: (index, groups PX, workgroups per group PR, rows per
// workgroup R, units per group U). hidden = PX * U; batches up to PR * R.
#define MLP_SHAPES(X)                                                   \
    X(0, 8, 32, 128, 32)   /* 32-256-1,  batch <= 4096 */             \
    X(1, 8, 32, 64, 32)    /* 32-256-1,  batch <= 2048 */             \
    X(2, 8, 32, 32, 32)    /* 32-256-1,  batch <= 1024 */             \
    X(3, 4, 32, 16, 64)    /* 32-256-1,  batch <= 512, four XCDs */   \
    X(4, 1, 16, 16, 256)   /* 32-256-1,  batch <= 256, one XCD */     \
    X(5, 8, 32, 32, 128)   /* 32-1024-1, batch <= 1024 */             \
    X(6, 8, 32, 16, 128)   /* 32-1024-1, batch <= 512  */             \
    X(7, 8, 32, 16, 64)    /* 32-512-1,  batch <= 512  */             \
    X(8, 2, 16, 16, 64)    /* 32-128-1,  batch <= 256, two XCDs */    \
    X(9, 1, 16, 16, 64)   /* 32-64-1,   batch <= 256, one XCD */     \
    X(10, 1, 8, 32, 32)    /* 32-32-1,   batch <= 256, one XCD */     \
    X(11, 4, 16, 16, 64)   /* 32-256-1,  batch <= 256, four XCDs */   \
    X(12, 2, 16, 16, 128)  /* 32-256-1,  batch <= 256, two XCDs */

#define MLP_SHAPE_TYPE(I, PX, PR, R, U) typedef Shape<PX, PR, R, U> Shape##I;
MLP_SHAPES(MLP_SHAPE_TYPE)
#undef MLP_SHAPE_TYPE

static const TrainPlan *all_plans(int *count) {
    static TrainPlan plans[32];
    static int n = 0;
    if (n == 0) {
#define MLP_SHAPE_PLAN(I, PX, PR, R, U) plans[n++] = plan_of<Shape##I>(I);
        MLP_SHAPES(MLP_SHAPE_PLAN)
#undef MLP_SHAPE_PLAN
    }
    *count = n;
    return plans;
}

// Modelled step time: MFMA work of one wave plus the exchange latencies
// (one exchange across XCDs when PX > 1, two inside one XCD).
static double plan_cost(const TrainPlan &pl) {
    const double mfma_cycles = 32.0 * 16.0 * pl.nuw * pl.rtw;
    const double compute = 2.0 * mfma_cycles / 2.4e9;
    return compute + (pl.px > 1 ? 1.5e-6 : 0.0) + 1.4e-6;
}

bool plan_train(int hidden, int64_t batch, TrainPlan *plan) {
    const char *force = getenv("MLP_PX");
    const int fpx = force ? atoi(force) : 0;
    const char *force_inst = getenv("MLP_INST");
    const int finst = force_inst ? atoi(force_inst) : -1;
    int n = 0;
    const TrainPlan *plans = all_plans(&n);
    bool found = false;
    double best_cost = 0.0;
    int64_t best_cap = 0;
    for (int i = 0; i < n; ++i) {
        const TrainPlan &pl = plans[i];
        const int64_t cap = (int64_t)pl.pr * pl.R;
        if (pl.px * pl.U != hidden || cap < batch) continue;
        if (fpx && pl.px != fpx) continue;
        if (finst >= 0 && pl.inst != finst) continue;
        // modelled cost first, then the tightest capacity (fewest idle rows)
        const double cst = plan_cost(pl);
        if (!found || cst < best_cost - 1e-12 || (cst < best_cost + 1e-12 && cap < best_cap)) {
            *plan = pl;
            best_cost = cst;
            best_cap = cap;
            found = true;
        }
    }
    return found;
}

size_t persist_words_xch() { return (size_t)2 * 32 * 8 * RMAX; }
size_t persist_words_rs(int hidden) { return (size_t)2 * 32 * ((size_t)hidden * 32 + 8 * 32); }
size_t persist_words_ag(int hidden) { return (size_t)2 * hidden * 33; }

hipError_t launch_train(Ctx &c, TrainArgs &a) {
    a.xch = c.xch;
    a.rs = c.rs;
    a.ag = c.ag;
    a.reg = c.ctl->reg;
    a.abort = &c.ctl->abort;
    a.err = &c.ctl->err;
    a.tag_base = c.tag_base;
    a.timeout_ticks = 200000000ull;   // 2 s
    const char *tr = getenv("MLP_TRACE");
    a.trace = (tr && (tr[0] == '1' || tr[0] == '2')) ? c.ctl->trace : nullptr;
    a.trace_all = (tr && tr[0] == '2') ? reinterpret_cast<uint64_t *>(c.slots) : nullptr;
    const char *fc = getenv("MLP_FORCE_COHERENT");
    a.force_coherent = (fc && fc[0] == '1') ? 1 : 0;
    // tags of the next call start past every tag this call can use
    c.tag_base += (uint32_t)(a.steps + 2);
    if (c.tag_base < 1) c.tag_base = 1;
    switch (a.plan.inst) {
#define MLP_SHAPE_CASE(I, PX, PR, R, U) \
    case I: return launch_shape<Shape##I>(c.stream, a);
        MLP_SHAPES(MLP_SHAPE_CASE)
#undef MLP_SHAPE_CASE
    }
    return hipErrorInvalidValue;
}

}  // namespace mlp
