// train_persistent.hip -- single-launch fused mini-batch SGD trainer for the
// d-h-1 ReLU/MSE network (paper Sec. III eqs. 11-19, d = 32), for gfx950.
//
// Decomposition (one workgroup per CU):
//   - the hidden units are split over PX groups of workgroups; each group lives
//     on one XCD (8 XCDs, one L2 each) and owns U = h/PX units;
//   - inside a group, PR workgroups split the rows of every mini-batch (R rows
//     each); every workgroup holds the group's W1 slice [32 x U] and W2 slice [U].
// A workgroup has four compute waves (one per SIMD, all on MFMA) and one loader
// wave that gathers the rows of later steps through the epoch permutation.
// One SGD step is:
//   1. Z1 = X W1 on fp32 MFMA (16x16x4) from the rows staged in LDS; ReLU mask
//      bits and the partial Ypred over the group's units stay in registers
//      (eqs. 11-13);
//   2. exchange A (across XCDs, PX-way): each wave sums the PX partial Ypred of
//      its rows in group order -> Ypred, residual, dZ2 = (2/n_b) r (eqs. 14-15);
//   3. P = X^T (dZ2 (.) [Z1 > 0]) on MFMA over the wave's rows; the wave
//      partials are summed in LDS (the first of two workgroup barriers per step);
//      dW1 = P diag(W2) and dW2_j = sum_k W1_kj P_kj then equal eqs. 16-18
//      (H_rj = [Z1_rj > 0] sum_k X_rk W1_kj);
//   4. exchange B (inside the XCD, reduce-scatter): the owner of each unit sums
//      its P column over the group's workgroups in a fixed order and applies
//      W -= lr dW (eq. 19);
//   5. exchange C (inside the XCD, all-gather): every workgroup loads the
//      updated slice into LDS (the second barrier publishes it, together with the
//      next step's rows).
// Exchanges use 64-bit words holding (fp32 value, 32-bit step tag). Writers
// never wait; readers load their words directly and reload any word whose tag
// is not yet current. Every sum runs in a fixed order, so results are bitwise
// reproducible and identical in every group that computes them. No
// floating-point atomics are used. The batch loss is reduced one step late by a
// single wave, off the critical path.
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

#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int NCW = 4;                  // compute waves per workgroup
constexpr int NTHR = 64 * (NCW + 1);    // plus one loader wave

// ---------------------------------------------------------------------------
// Shapes
// ---------------------------------------------------------------------------

template <int PX_, int PR_, int R_, int U_>
struct Shape {
    static constexpr int PX = PX_, PR = PR_, R = R_, U = U_;
    static constexpr int H = PX * U;                       // hidden units
    static constexpr int NR = R / 16, NU = U / 16;         // row / unit tiles
    static constexpr int WR = NR >= 4 ? 4 : NR;            // waves along rows
    static constexpr int WU = NCW / WR;                    // waves along units
    static constexpr int RTW = NR / WR;                    // row tiles per wave (contiguous)
    static constexpr int NUW = NU / WU;                    // unit tiles per wave (stride WU)
    static constexpr int NRW = RTW * 16;                   // rows per wave
    static constexpr int UPW = U / PR;                     // units owned per workgroup
    static constexpr int NPAIR = UPW * 32;                 // owned (k, unit) pairs
    static constexpr int OWN_T = NPAIR >= 256 ? 256 : (NPAIR >= 64 ? NPAIR : 64);
    static constexpr int SPLIT = NPAIR >= 64 ? 1 : 64 / NPAIR;   // partial-range splits
    static constexpr int TPS = OWN_T / SPLIT;              // owner threads per split
    static constexpr int PPT = NPAIR / TPS;                // pairs per owner thread
    static constexpr int LPS = PR / SPLIT;                 // partials per split
    static constexpr int ASPL0 = 64 / NRW;                 // exchange-A lane splits
    static constexpr int ASPL = ASPL0 < PX ? ASPL0 : PX;
    static constexpr int APPS = PX / ASPL;                 // peers per exchange-A lane
    static_assert(ASPL == 1 || ASPL == 2 || ASPL == 4, "exchange-A lane splits");
    static constexpr int XS = 36;                          // X tile row stride (floats)
    static constexpr int WS = 36;                          // weight slice row stride
    static constexpr int PS = U + 1;                       // P partial row stride
    static constexpr int RSW = 32 * U;                     // exchange-B words per workgroup
    static constexpr int GBW = (PR * RSW + PR + 31) / 32 * 32;   // exchange-B words per group
    static constexpr int RPL = R / 8;                      // rows per loader lane
    // LDS carve-up, in floats
    static constexpr int O_X = 0;                          // [2][R][XS] staged rows
    static constexpr int O_Y = O_X + 2 * R * XS;           // [2][R]
    static constexpr int O_YP = O_Y + 2 * R;               // [WU][R] partial Ypred
    static constexpr int O_G = O_YP + WU * R;              // [NCW][NRW] dZ2 per wave
    static constexpr int O_P = O_G + NCW * NRW;            // [WR][32][PS] P partials
    static constexpr int O_WSL = O_P + WR * 32 * PS;       // [U][WS] weight slice
    static constexpr int O_SSE = O_WSL + U * WS;           // [NCW]
    static constexpr int LDS_FLOATS = O_SSE + NCW;

    static_assert(R % 16 == 0 && U % 16 == 0, "tiles");
    static_assert(WR * WU == NCW && NR % WR == 0 && NU % WU == 0, "wave split");
    static_assert(NUW >= 1 && RTW >= 1 && NUW * RTW <= 8, "mask bits");
    static_assert(NRW == 16 || NRW == 32 || NRW == 64, "exchange-A lanes");
    static_assert(U % PR == 0 && UPW >= 1 && NPAIR % TPS == 0 && PR % SPLIT == 0, "ownership");
    static_assert(RSW % 256 == 0, "exchange-B stores");
    static_assert(R <= RMAX && R <= 128, "rows");
    static_assert(PX == 1 || PX == 2 || PX == 4 || PX == 8, "groups");
    static_assert(PR >= 1 && PR <= 32, "workgroups per group");
    static_assert(O_WSL % 4 == 0 && O_G % 4 == 0, "float4 alignment");
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

// Order LDS traffic between the lanes of one wave (no workgroup barrier).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Read a field of the kernel argument block at its use, straight from the
// kernarg segment: the load is not hoisted to the kernel entry, so arguments
// needed only off the hot path hold no registers through the step loop.
typedef const char __attribute__((address_space(4))) *kernarg_ptr;
template <class T>
__device__ __forceinline__ T cold_at(size_t off) {
    kernarg_ptr base = (kernarg_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(base));
    return *(const T __attribute__((address_space(4))) *)(base + off);
}
#define COLD(field) cold_at<decltype(TrainArgs::field)>(offsetof(TrainArgs, field))

// Waits of one lane. A wait that outlives the limit raises the kernel-wide
// abort word and the workgroup's abort stamp (step + 1, in LDS); every later
// wait of the step returns at once, and all waves leave the step loop together
// at the top of the next step.
struct Waiter {
    int *stamp;
    int step;
    bool aborted;

    __device__ __forceinline__ void check(uint64_t deadline) {
        int32_t *abort = COLD(abort);
        if (__hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
            aborted = true;
        } else if (now_ticks() > deadline) {
            __hip_atomic_store(COLD(err), (int32_t)MLP_ERR_TIMEOUT_CODE, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            aborted = true;
        }
        if (aborted) *stamp = step + 1;
    }
    // w[i] was loaded from p + i * STRIDE; reload the words until every tag is
    // current. The retry path rebuilds its addresses from p, so no per-word
    // address stays live in registers.
    template <int N, int STRIDE>
    __device__ __forceinline__ void settle(uint64_t (&w)[N], const uint64_t *p, uint32_t tag) {
        uint32_t spins = 0;
        uint64_t deadline = 0;
        while (true) {
            uint32_t bad = 0;
#pragma unroll
            for (int i = 0; i < N; ++i) bad |= tag_of(w[i]) ^ tag;
            if (bad == 0 || aborted) break;
            if (spins == 0) deadline = now_ticks() + COLD(timeout_ticks);
            if ((++spins & 63u) == 0) {
                check(deadline);
                if (aborted) break;
            }
            __builtin_amdgcn_s_sleep(1);
            const uint64_t *q = p;
            asm volatile("" : "+v"(q));
            if constexpr (N == 1) {
                w[0] = ld_dev(q);
            } else {
#pragma unroll
                for (int i = 0; i < N; ++i) w[i] = ld_dev(q + i * STRIDE);
            }
        }
    }
};

// C words per thread of the all-gathered weight slice ([unit][33] words, word
// i at src + 256 q for i = i0 + 256 q) into the LDS slice ([unit][WS] floats).
template <int C, int WS>
__device__ __forceinline__ void gather_slice(Waiter &wt, const uint64_t *src, float *Wsl, int i0,
                                             uint32_t tag) {
    uint64_t w[C];
#pragma unroll
    for (int q = 0; q < C; ++q) w[q] = ld_dev(src + 256 * q);
    wt.settle<C, 256>(w, src, tag);
#pragma unroll
    for (int q = 0; q < C; ++q) {
        const int i = i0 + 256 * q, jl = i / 33, k = i - jl * 33;
        Wsl[jl * WS + k] = val_of(w[q]);
    }
}

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
// Butterfly sums (every lane gets the total, in a fixed order).
__device__ __forceinline__ float sum32(float v) {
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 1, 64);
    return v;
}
__device__ __forceinline__ float sum64(float v) {
    v = sum32(v);
    return v + __shfl_xor(v, 32, 64);
}

// (epoch, step within the epoch) of a step
struct Pos {
    int e, sb;
    __device__ __forceinline__ void advance(int spe) {
        if (++sb == spe) {
            sb = 0;
            ++e;
        }
    }
};

// Optional phase timestamps (s_memrealtime, 100 MHz): workgroup (0, 0) for the
// first TRACE_STEPS steps, or every workgroup for steps [16, 24).
constexpr int TRACE_STEPS = 48;
constexpr int TRACE_ALL_FIRST = 16, TRACE_ALL_STEPS = 8;
#define TRACE(ph)                                                                          \
    do {                                                                                   \
        if constexpr (TR)                                                                  \
        if (a.trace && tid == 0 && gx == 0 && gb == 0 && s < TRACE_STEPS)                  \
            a.trace[s * 8 + (ph)] = now_ticks();                                           \
        if constexpr (TR)                                                                  \
        if (a.trace_all && tid == 0 && s >= TRACE_ALL_FIRST &&                             \
            s < TRACE_ALL_FIRST + TRACE_ALL_STEPS)                                         \
            a.trace_all[((gx * S::PR + gb) * TRACE_ALL_STEPS + (s - TRACE_ALL_FIRST)) * 8 + \
                        (ph)] = now_ticks();                                               \
    } while (0)

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
// Compute wave w = wr + wu * WR takes row tiles [wr * RTW, (wr + 1) * RTW) and
// unit tiles {wu + i * WU}. Wave NCW is the loader. Both kinds of wave pass the
// same workgroup barriers: one before the loop, then per step [one more when
// WU > 1,] "P partials ready" and "next step ready".
template <class S, bool TR>
__global__ __launch_bounds__(NTHR) void k_train(const TrainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int s_flags[8];   // 0: group x, 1: rank b, 2: plain local stores, 3: abort stamp, 4: active

    constexpr int R = S::R, U = S::U, PR = S::PR, PX = S::PX, H = S::H;
    constexpr int WR = S::WR, WU = S::WU, NUW = S::NUW, RTW = S::RTW, NRW = S::NRW;
    constexpr int UPW = S::UPW, NPAIR = S::NPAIR, XS = S::XS, WS = S::WS, PS = S::PS;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lq = lane >> 4, li = lane & 15;   // lane group (0..3) and index in group

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
    const int gx = __builtin_amdgcn_readfirstlane(s_flags[0]);
    const int gb = __builtin_amdgcn_readfirstlane(s_flags[1]);
    const bool plain = __builtin_amdgcn_readfirstlane(s_flags[2]) != 0;
    const bool run = __builtin_amdgcn_readfirstlane(s_flags[4]) != 0 &&
                     __builtin_amdgcn_readfirstlane(s_flags[3]) == 0;
    __syncthreads();
    if (tid == 0) s_flags[3] = 0;   // from here on: the abort stamp

    float *Xall = lds + S::O_X;     // [2][R][XS]
    float *Yall = lds + S::O_Y;     // [2][R]
    float *Ypart = lds + S::O_YP;   // [WU][R]
    float *Gw = lds + S::O_G;       // [NCW][NRW]
    float *Pred = lds + S::O_P;     // [WR][32][PS]
    float *Wsl = lds + S::O_WSL;    // [U][WS]
    float *SseW = lds + S::O_SSE;   // [NCW]

    const int steps = (int)a.steps;
    const int spe = (int)((a.n + a.batch - 1) / a.batch);
    const int batch = (int)a.batch;
    const int tail = (int)(a.n - (int64_t)(spe - 1) * a.batch);

    if (run) {
        // ---- the group's weight slice (all waves) ---------------------------------
        for (int i = tid; i < U * 33; i += NTHR) {
            const int jl = i / 33, k = i - jl * 33;
            const int ug = gx * U + jl;
            Wsl[jl * WS + k] = k < 32 ? COLD(W1)[k * H + ug] : COLD(W2)[ug];
        }
        Waiter wt{&s_flags[3], 0, false};

        if (wave < NCW) {
            // ================= compute waves =================================
            const int wr = wave % WR, wu = wave / WR;
            const bool owner = tid < S::OWN_T;
            const int osplit = tid / S::TPS, ot = tid % S::TPS;
            float ow1[S::PPT], ow2[S::PPT];   // master copy of the owned pairs
            if (owner) {
#pragma unroll
                for (int q = 0; q < S::PPT; ++q) {
                    const int p = ot + S::TPS * q, jl = p >> 5, k = p & 31;
                    const int ug = gx * U + gb * UPW + jl;
                    ow1[q] = COLD(W1)[k * H + ug];
                    ow2[q] = COLD(W2)[ug];
                }
            }
            // the loss is reduced one step late by wave 1 of workgroup (0, 0)
            const bool lossw = gx == 0 && gb == 0 && wave == 1;
            double epoch_sse = 0.0;
            Pos cur{0, 0}, prev{0, 0};
            int nb_prev = 1;
            int done = 0;
            const int rl = lane % NRW;             // row within the wave's rows
            const int rw = wr * NRW + rl;          // row within the workgroup
            __syncthreads();                       // weights and the first rows staged

            for (int s = 0; s < steps; ++s) {
                {
                    const int st = s_flags[3];
                    if (st != 0 && st <= s) break;   // a wave aborted in an earlier step
                }
                wt.step = s;
                const uint32_t tag = a.tag_base + (uint32_t)s;
                const int par = s & 1;
                const int nb = cur.sb == spe - 1 ? tail : batch;
                const int rc = nb - gb * R;        // rows of this workgroup in the batch (may be <= 0)
                const float scale = 2.0f / (float)nb;
                const float *Xb = Xall + par * R * XS;
                const float *Yb = Yall + par * R;
                uint64_t *rsg = a.rs + (size_t)(par * PX + gx) * S::GBW;
                TRACE(0);

                // deferred loss: issue the loads of the previous step's SSE partials
                const uint32_t tag_prev = tag - 1;
                const uint64_t *sse_prev = a.rs + (size_t)((par ^ 1) * PX) * S::GBW + PR * S::RSW +
                                           (lane < PR ? lane : 0);
                uint64_t sw[1] = {pack(0.f, tag_prev)};
                if (lossw && s > 0 && lane < PR) sw[0] = ld_dev(sse_prev);

                // ---- 1. forward: Z1 tiles, mask bits, partial Ypred ---------------
                float w1b[NUW][8], w2v[NUW];
#pragma unroll
                for (int u = 0; u < NUW; ++u) {
                    const float *wp = Wsl + ((wu + u * WU) * 16 + li) * WS + 8 * lq;
                    const float4 a0 = *reinterpret_cast<const float4 *>(wp);
                    const float4 a1 = *reinterpret_cast<const float4 *>(wp + 4);
                    w1b[u][0] = a0.x; w1b[u][1] = a0.y; w1b[u][2] = a0.z; w1b[u][3] = a0.w;
                    w1b[u][4] = a1.x; w1b[u][5] = a1.y; w1b[u][6] = a1.z; w1b[u][7] = a1.w;
                    w2v[u] = Wsl[((wu + u * WU) * 16 + li) * WS + 32];
                }
                uint32_t mbits = 0;   // bit (i*NUW + u)*4 + v
#pragma unroll
                for (int i = 0; i < RTW; ++i) {
                    const int tile = wr * RTW + i;
                    const float *xr = Xb + (tile * 16 + li) * XS + 8 * lq;
                    const float4 xa = *reinterpret_cast<const float4 *>(xr);
                    const float4 xb = *reinterpret_cast<const float4 *>(xr + 4);
                    const float xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
                    f4 acc[NUW];
#pragma unroll
                    for (int u = 0; u < NUW; ++u) acc[u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int t = 0; t < 8; ++t)
#pragma unroll
                        for (int u = 0; u < NUW; ++u)
                            acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[t], w1b[u][t], acc[u], 0, 0, 0);
                    float yp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int u = 0; u < NUW; ++u)
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const float z = acc[u][v];
                            const bool on = z > 0.0f;                       // ReLU'(z) = [z > 0]
                            mbits |= (on ? 1u : 0u) << ((i * NUW + u) * 4 + v);
                            yp[v] = fmaf(on ? z : 0.0f, w2v[u], yp[v]);     // eqs. 12-13
                        }
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float sv = row16_sum(yp[v]);
                        if (li == 15) Ypart[wu * R + tile * 16 + 4 * lq + v] = sv;
                    }
                }
                if constexpr (WU > 1)
                    __syncthreads();   // partial Ypred of the unit waves
                else
                    wave_sync();
                float yv = 0.f;
#pragma unroll
                for (int w = 0; w < WU; ++w) yv += Ypart[w * R + rw];
                TRACE(1);

                // ---- 2. exchange A: partial Ypred across groups ------------------
                if constexpr (PX > 1) {
                    uint64_t *xa = a.xch + (size_t)((par * PR + gb) * PX) * RMAX;
                    if (wu == 0 && lane < NRW) st_dev(xa + gx * RMAX + rw, pack(yv, tag));
                    const int sp = (lane / NRW) % S::ASPL;
                    const uint64_t *src = xa + (size_t)(sp * S::APPS) * RMAX + rw;
                    uint64_t w[S::APPS];
#pragma unroll
                    for (int x = 0; x < S::APPS; ++x) w[x] = ld_dev(src + x * RMAX);
                    wt.settle<S::APPS, RMAX>(w, src, tag);
                    float t = 0.f;
#pragma unroll
                    for (int x = 0; x < S::APPS; ++x) t += val_of(w[x]);
                    if constexpr (S::ASPL >= 2) t += __shfl_xor(t, NRW, 64);
                    if constexpr (S::ASPL >= 4) t += __shfl_xor(t, 2 * NRW, 64);
                    yv = t;
                }
                TRACE(2);

                // residual, dZ2 (eqs. 14-15), SSE of the wave's rows
                {
                    const float res = yv - Yb[rw];
                    const bool in = rw < rc;
                    const float g = in ? scale * res : 0.0f;
                    const float r2 = (in && lane < NRW && wu == 0) ? res * res : 0.0f;
                    const float sse = sum64(r2);
                    if (lane == 0) SseW[wave] = sse;
                    if (lane < NRW) Gw[wave * NRW + rl] = g;
                    wave_sync();
                }

                // ---- 3. backward: P = X^T (dZ2 (.) mask) -------------------------
                f4 pacc[2][NUW];
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int u = 0; u < NUW; ++u) pacc[kt][u] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i = 0; i < RTW; ++i) {
                    const int tile = wr * RTW + i;
                    const float4 g4 = *reinterpret_cast<const float4 *>(Gw + wave * NRW + 16 * i + 4 * lq);
                    const float gv[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float *xr = Xb + (tile * 16 + 4 * lq + v) * XS + li;
                        const float xt0 = xr[0], xt1 = xr[16];
#pragma unroll
                        for (int u = 0; u < NUW; ++u) {
                            const bool on = (mbits >> ((i * NUW + u) * 4 + v)) & 1u;
                            const float gm = on ? gv[v] : 0.0f;     // dZ2 (.) ReLU'(Z1)
                            pacc[0][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xt0, gm, pacc[0][u], 0, 0, 0);
                            pacc[1][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xt1, gm, pacc[1][u], 0, 0, 0);
                        }
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

                // deferred loss of the previous step (its words are long written)
                if (lossw && s > 0) {
                    wt.settle<1, 0>(sw, sse_prev, tag_prev);
                    const float sse = sum64(lane < PR ? val_of(sw[0]) : 0.0f);
                    if (lane == 0) {
                        const float L = sse / (float)nb_prev;               // eq. 14
                        float *lo = COLD(loss), *sl = COLD(step_loss), *el = COLD(epoch_loss);
                        if (lo) lo[0] = L;
                        if (sl) sl[s - 1] = L;
                        if (prev.sb == 0) epoch_sse = 0.0;
                        epoch_sse += (double)sse;
                        if (el) el[prev.e] = (float)(epoch_sse * (double)COLD(inv_n));
                    }
                }
                __syncthreads();   // P partials and SSE of every wave in LDS
                TRACE(3);

                // ---- 4. exchange B: reduce-scatter of P inside the group ---------
                // word (ul, k) of this workgroup goes to owner o = ul / UPW at
                // rsg + (o * PR + gb) * NPAIR + (ul % UPW) * 32 + k
#pragma unroll
                for (int i0 = 0; i0 < S::RSW; i0 += 256) {
                    const int i = i0 + tid;
                    const int ul = i >> 5, k = i & 31;
                    float v = 0.f;
#pragma unroll
                    for (int w = 0; w < WR; ++w) v += Pred[(w * 32 + k) * PS + ul];
                    const int o = ul / UPW, jl = ul - o * UPW;
                    st_loc(rsg + (size_t)(o * PR + gb) * NPAIR + jl * 32 + k, pack(v, tag), plain);
                }
                if (tid == 0) {
                    float v = 0.f;
#pragma unroll
                    for (int w = 0; w < WR; ++w) v += SseW[w];
                    st_loc(rsg + PR * S::RSW + gb, pack(gx == 0 ? v : 0.f, tag), plain);
                }
                if (owner) {
                    const uint64_t *ob = rsg + (size_t)(gb * PR + osplit * S::LPS) * NPAIR;
                    uint64_t w[S::PPT][S::LPS];
#pragma unroll
                    for (int q = 0; q < S::PPT; ++q)
#pragma unroll
                        for (int b = 0; b < S::LPS; ++b)
                            w[q][b] = ld_dev(ob + b * NPAIR + ot + S::TPS * q);
                    float pk[S::PPT];
#pragma unroll
                    for (int q = 0; q < S::PPT; ++q) {
                        wt.settle<S::LPS, NPAIR>(w[q], ob + ot + S::TPS * q, tag);
                        float t = 0.f;
#pragma unroll
                        for (int b = 0; b < S::LPS; ++b) t += val_of(w[q][b]);
                        if constexpr (S::SPLIT == 2) t += __shfl_xor(t, 32, 64);
                        pk[q] = t;
                    }
                    TRACE(4);
                    // ---- update the owned units (eq. 19) or emit gradients ------
                    uint64_t *agg = a.ag + (size_t)(par * PX + gx) * (U * 33);
#pragma unroll
                    for (int q = 0; q < S::PPT; ++q) {
                        const int p = ot + S::TPS * q, jl = p >> 5, k = p & 31;
                        const int ug = gx * U + gb * UPW + jl;
                        const float w1 = ow1[q], w2 = ow2[q];
                        const float dw1 = w2 * pk[q];                      // dW1_kj = W2_j P_kj
                        const float dw2 = sum32(w1 * pk[q]);               // dW2_j = sum_k W1_kj P_kj
                        if (a.mode == 1) {
                            if (osplit == 0) {
                                COLD(dW1)[k * H + ug] = dw1;
                                if (k == 0) COLD(dW2)[ug] = dw2;
                            }
                        } else {
                            ow1[q] = w1 - a.lr * dw1;
                            ow2[q] = w2 - a.lr * dw2;
                            if (osplit == 0) {
                                st_loc(agg + (gb * UPW + jl) * 33 + k, pack(ow1[q], tag), plain);
                                if (k == 0) st_loc(agg + (gb * UPW + jl) * 33 + 32, pack(ow2[q], tag), plain);
                            }
                        }
                    }
                    TRACE(5);
                }

                // ---- 5. exchange C: all-gather the group's updated slice ---------
                if (a.mode == 0) {
                    // at most CH words per thread in flight, to bound registers
                    const uint64_t *agg = a.ag + (size_t)(par * PX + gx) * (U * 33);
                    constexpr int NW = U * 33, FULL = NW / 256, REST = NW % 256;
                    constexpr int CH = FULL < 17 ? FULL : 16;
                    constexpr int NCH = (FULL + CH - 1) / CH;
                    uint64_t wt1[1] = {pack(0.f, tag)};
                    if (REST > 0 && tid < REST) wt1[0] = ld_dev(agg + 256 * FULL + tid);
#pragma unroll
                    for (int c = 0; c < NCH - 1; ++c)
                        gather_slice<CH, WS>(wt, agg + tid + 256 * CH * c, Wsl, tid + 256 * CH * c, tag);
                    gather_slice<FULL - (NCH - 1) * CH, WS>(wt, agg + tid + 256 * CH * (NCH - 1), Wsl,
                                                            tid + 256 * CH * (NCH - 1), tag);
                    if (REST > 0 && tid < REST) {
                        wt.settle<1, 0>(wt1, agg + 256 * FULL + tid, tag);
                        const int i = 256 * FULL + tid, jl = i / 33, k = i - jl * 33;
                        Wsl[jl * WS + k] = val_of(wt1[0]);
                    }
                }
                TRACE(6);
                prev = cur;
                nb_prev = nb;
                cur.advance(spe);
                done = s + 1;
                __syncthreads();   // next step's rows staged, weight slice updated
            }

            // ---- after the loop -----------------------------------------------------
            const bool aborted = s_flags[3] != 0;
            if (!aborted && done > 0 && lossw) {
                // loss of the last step
                const uint32_t tag_last = a.tag_base + (uint32_t)(done - 1);
                const uint64_t *sse_last = a.rs + (size_t)(((done - 1) & 1) * PX) * S::GBW +
                                           PR * S::RSW + (lane < PR ? lane : 0);
                uint64_t swl[1] = {pack(0.f, tag_last)};
                if (lane < PR) swl[0] = ld_dev(sse_last);
                wt.settle<1, 0>(swl, sse_last, tag_last);
                const float sse = sum64(lane < PR ? val_of(swl[0]) : 0.0f);
                if (lane == 0) {
                    const float L = sse / (float)nb_prev;
                    float *lo = COLD(loss), *sl = COLD(step_loss), *el = COLD(epoch_loss);
                    if (lo) lo[0] = L;
                    if (sl) sl[done - 1] = L;
                    if (prev.sb == 0) epoch_sse = 0.0;
                    epoch_sse += (double)sse;
                    if (el) {
                        el[prev.e] = (float)(epoch_sse * (double)COLD(inv_n));
                        for (int e = prev.e + 1; e < COLD(epochs); ++e) el[e] = 0.0f;
                    }
                }
            }
            if (a.mode == 0 && owner && osplit == 0) {
#pragma unroll
                for (int q = 0; q < S::PPT; ++q) {
                    const int p = ot + S::TPS * q, jl = p >> 5, k = p & 31;
                    const int ug = gx * U + gb * UPW + jl;
                    COLD(W1)[k * H + ug] = ow1[q];
                    if (k == 0) COLD(W2)[ug] = ow2[q];
                }
            }
        } else {
            // ================= loader wave ====================================
            // Indices are loaded two steps ahead and rows one step ahead into
            // registers; a step's rows are written to LDS during the step before.
            constexpr int RPL = S::RPL;
            const int lc = lane & 7, lr0 = lane >> 3;   // float4 chunk, first row
            const int64_t row0 = (int64_t)gb * R;
            int32_t pidx[RPL];
            float4 pfx[RPL];
            float pfy[RPL];
            auto fetch_idx = [&](const Pos &ps) {
                const int64_t off = (int64_t)ps.sb * COLD(batch);
                const int32_t *perm = COLD(perm);
                const int64_t n = COLD(n);
#pragma unroll
                for (int j = 0; j < RPL; ++j) {
                    int64_t pos = off + row0 + lr0 + 8 * j;
                    if (perm) {
                        pos = pos < n ? pos : n - 1;                // always a valid address
                        pidx[j] = perm[(int64_t)ps.e * n + pos];
                    } else {
                        pidx[j] = (int32_t)pos;
                    }
                }
            };
            auto fetch_rows = [&](const Pos &ps) {
                const int nbr = ps.sb == spe - 1 ? tail : batch;
                const int64_t rcl = nbr - row0;
                const float *X = COLD(X), *Y = COLD(Y);
                const int64_t n_rows = COLD(n_rows);
#pragma unroll
                for (int j = 0; j < RPL; ++j) {
                    const int r = lr0 + 8 * j;
                    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                    float y = 0.f;
                    if (r < rcl) {
                        int64_t row = pidx[j];
                        if (row < 0 || row >= n_rows) {
                            __hip_atomic_store(COLD(err), (int32_t)MLP_ERR_INDEX, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                            row = 0;
                        }
                        v = *reinterpret_cast<const float4 *>(X + row * D_IN + 4 * lc);
                        if (lc == 0) y = Y[row];
                    }
                    pfx[j] = v;
                    pfy[j] = y;
                }
            };
            auto stage = [&](int buf) {
                float *Xd = Xall + buf * R * XS;
                float *Yd = Yall + buf * R;
#pragma unroll
                for (int j = 0; j < RPL; ++j) {
                    const int r = lr0 + 8 * j;
                    *reinterpret_cast<float4 *>(Xd + r * XS + 4 * lc) = pfx[j];
                    if (lc == 0) Yd[r] = pfy[j];
                }
            };
            Pos q1{0, 0};
            if (steps > 0) {
                fetch_idx(q1);
                fetch_rows(q1);
                stage(0);
            }
            q1.advance(spe);
            Pos q2 = q1;
            q2.advance(spe);
            if (steps > 1) {
                fetch_idx(q1);
                fetch_rows(q1);
            }
            if (steps > 2) fetch_idx(q2);
            __syncthreads();   // weights and the first rows staged

            for (int s = 0; s < steps; ++s) {
                {
                    const int st = s_flags[3];
                    if (st != 0 && st <= s) break;
                }
                if constexpr (WU > 1) __syncthreads();
                // registers hold the rows of step s+1 and the indices of step s+2
                // (position q2)
                if (s + 1 < steps) stage((s + 1) & 1);
                Pos q3 = q2;
                q3.advance(spe);
                if (s + 2 < steps) fetch_rows(q2);
                if (s + 3 < steps) fetch_idx(q3);
                q2 = q3;
                __syncthreads();   // P partials ready
                __syncthreads();   // next step ready
            }
        }
    }

    // ---- teardown: the last workgroup out clears the registration counters ------
    __syncthreads();
    if (tid == 0) {
        const int fin = __hip_atomic_fetch_add(&a.reg[10], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if (fin == (int)gridDim.x - 1) {
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
    const void *fn = (a.trace || a.trace_all) ? reinterpret_cast<const void *>(&k_train<S, true>)
                                              : reinterpret_cast<const void *>(&k_train<S, false>);
    return hipLaunchCooperativeKernel(fn,
                                      dim3(a.plan.grid), dim3(NTHR), args, (unsigned)a.plan.lds,
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
    p.rs_stride = S::GBW;
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
    X(9, 1, 16, 16, 64)    /* 32-64-1,   batch <= 256, one XCD */     \
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

// Modelled step time: MFMA work of one wave (forward and backward, 32 cycles
// per 16x16x4 fp32 MFMA) plus the exchange latencies (one across XCDs when
// PX > 1, two inside one XCD).
static double plan_cost(const TrainPlan &pl) {
    const double mfma_cycles = 32.0 * 16.0 * pl.nuw * pl.rtw;
    const double compute = mfma_cycles / 2.4e9;
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
// two parities x up to 8 groups x (32 workgroups x 32 U words + 32 loss words)
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
