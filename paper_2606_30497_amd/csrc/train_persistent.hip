// train_persistent.hip -- single-launch fused mini-batch SGD trainer for the
// d-h-1 ReLU/MSE network (paper Sec. III eqs. 11-19, d = 32), for gfx950.
//
// Decomposition (one workgroup per CU):
//   - the hidden units are split over PX groups of workgroups; each group lives
//     on one XCD (8 XCDs, one L2 each) and owns U = h/PX units;
//   - inside a group, PR workgroups split the rows of every mini-batch (R rows
//     each); every workgroup holds the group's W1 slice [32 x U] and W2 slice [U].
// A workgroup has four compute waves (one per SIMD, all on MFMA) and two loader
// waves that gather the rows of later steps through the epoch permutation (one
// loader wave alone is limited by how fast it can issue the gathers).
// One SGD step is:
//   1. Z1 = X W1 on MFMA from the rows staged in LDS; ReLU mask bits and the
//      partial Ypred over the group's units stay in registers (eqs. 11-13);
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
// Both contractions are fp32 products computed on bf16 MFMA (16x16x32; 16x16x16
// for the backward of 16-row waves): every fp32 operand x is split into three
// bf16 parts x = x0 + x1 + x2 (each part the bf16 rounding of what the previous
// ones leave: |x1| <= 2^-8 |x|, |x2| <= 2^-16 |x|, and the three sum to x
// exactly while no part underflows), and of the nine part products the six
// with i + j <= 2 are accumulated in fp32, smallest first. The three dropped
// ones stay below about 2^-23 |a b| together (twice fp32's unit roundoff), so
// each product keeps fp32 accuracy, in about 2.5 times fewer MFMA cycles than
// on fp32 MFMA
// (8192 multiply-adds: six 16x16x32 bf16 MFMAs of about 17 cycles, against
// eight 16x16x4 fp32 ones of 32). bf16 MFMAs also leave the SIMD to the other
// waves (fp32 MFMAs hold off their issue). The loader waves split the rows they
// stage; the owners split the weights they update and publish the parts.
// Exchanges use 64-bit words holding (32-bit payload, 32-bit step tag): an fp32
// value, or, for the W1 words of exchange C, one bf16 part of two adjacent
// inputs. Writers
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
#include "lanes.h"
#include "mlp_internal.h"
#include "tags.h"

namespace mlp {

constexpr int NCW = 4;                  // compute waves per workgroup
constexpr int NLW = 2;                  // loader waves
constexpr int NTHR = 64 * (NCW + NLW);  // threads per workgroup

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
    static constexpr int NPAIR = UPW * 32;                 // owned (k, unit) words
    static constexpr int KP = NPAIR / 2;                   // owned (k pair, unit) items
    static constexpr int KPW = KP / 4 > 16 ? KP / 4 : 16;  // k pairs per owner wave
    static constexpr int NWO = KP / KPW;                   // owner waves
    static constexpr int OWN_T = 64 * NWO;                 // owner threads
    static constexpr int SG = 64 / KPW;                    // source groups in an owner wave
    static constexpr int LPS = PR / SG;                    // sources per owner lane
    static_assert(KP % 16 == 0 && KPW * NWO == KP && NWO >= 1 && NWO <= NCW && KPW <= 64 &&
                      PR % SG == 0 && (SG == 1 || SG == 2 || SG == 4), "ownership");
    static constexpr int XRS = 40;                         // bf16 row stride of a staged X part
    static constexpr int WPS = 40;                         // bf16 row stride of a W1 part (per unit)
    static constexpr int CW = 49 * U;                      // exchange-C words per group: [3][U][16] + [U]
    static constexpr int NPW = 3 * U / 32;                 // exchange-C word pairs per compute thread
    static constexpr int CHC = NPW <= 8 ? NPW : (NPW % 8 == 0 ? 8 : 6);   // of them in flight at once
    static constexpr int PS = 36;                          // P partial row stride (per unit, k inner)
    static constexpr int RSW = 32 * U;                     // exchange-B words per workgroup
    static constexpr int GBW = (PR * RSW + PR + 31) / 32 * 32;   // exchange-B words per group
    static constexpr int RPL = R / (8 * NLW);              // rows per loader lane
    // LDS carve-up, in bytes
    static constexpr int B_XR = 0;                               // [2][3][R][XRS] bf16: staged rows, split
    static constexpr int B_WP = B_XR + 2 * 3 * R * XRS * 2;      // [3][U][WPS] bf16: W1 slice, split
    static constexpr int B_W2 = B_WP + 3 * U * WPS * 2;          // [U] float: W2 slice
    static constexpr int B_Y = B_W2 + U * 4;                     // [2][R] float
    static constexpr int B_YP = B_Y + 2 * R * 4;                 // [WU][R] partial Ypred
    static constexpr int B_P = B_YP + WU * R * 4;                // [WR][U][PS] P partials
    static constexpr int B_SSE = B_P + WR * U * PS * 4;          // [NCW]
    static constexpr int LDS_BYTES = B_SSE + NCW * 4;

    static_assert(R % 16 == 0 && U % 16 == 0, "tiles");
    static_assert(WR * WU == NCW && NR % WR == 0 && NU % WU == 0, "wave split");
    static_assert(NUW >= 1 && RTW >= 1 && NUW * RTW <= 8, "mask bits");
    static_assert(NRW == 16 || NRW == 32 || NRW == 64, "exchange-A lanes");
    static_assert(U % PR == 0 && UPW >= 1, "units per workgroup");
    static_assert(RSW % 512 == 0, "exchange-B stores");
    static_assert(R <= RMAX && R <= 128, "rows");
    static_assert(PX == 1 || PX == 2 || PX == 4 || PX == 8, "groups");
    static_assert(PR >= 1 && PR <= 32, "workgroups per group");
    static_assert(B_WP % 16 == 0 && B_W2 % 16 == 0 && B_P % 16 == 0, "LDS alignment");
    static_assert(NPW * 256 * 2 == 48 * U && NPW % CHC == 0 && U / 2 <= 256, "exchange-C pairs");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS");
    static_assert(RTW == 1 || RTW == 2, "backward K blocks");
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

// Exchange words live in three buffers addressed through buffer resources
// (32-bit byte offsets). A load outside a buffer returns 0, which never carries a
// current tag, so a wrong offset shows up as a timeout, not as a stray access.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef int i2v __attribute__((ext_vector_type(2)));
typedef int i4v __attribute__((ext_vector_type(4)));
constexpr int CPOL_SC1 = 16;   // cache policy: device-coherent (sc1)

__device__ __forceinline__ rsrc_t make_rsrc(void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)bytes, 0x00020000);
}
struct W2 {   // two adjacent tagged words
    uint64_t a, b;
};
__device__ __forceinline__ uint64_t join(int lo, int hi) {
    return (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32);
}
// device-coherent loads of one / two adjacent words
__device__ __forceinline__ uint64_t ld1(rsrc_t r, uint32_t off) {
    const i2v v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, CPOL_SC1);
    return join(v.x, v.y);
}
__device__ __forceinline__ W2 ld2(rsrc_t r, uint32_t off) {
    const i4v v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CPOL_SC1);
    return W2{join(v.x, v.y), join(v.z, v.w)};
}
// store of one word: device-coherent (dev) or plain (lands in the XCD's L2)
__device__ __forceinline__ void st1(rsrc_t r, uint32_t off, uint64_t w, bool dev) {
    const i2v v = {(int)(uint32_t)w, (int)(uint32_t)(w >> 32)};
    if (dev)
        __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, CPOL_SC1);
    else
        __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}
// store of two adjacent words (16-byte aligned) in one 16-byte store; a reader
// checks the tag of each 8-byte word on its own
__device__ __forceinline__ void st2(rsrc_t r, uint32_t off, uint64_t w0, uint64_t w1, bool dev) {
    const i4v v = {(int)(uint32_t)w0, (int)(uint32_t)(w0 >> 32), (int)(uint32_t)w1,
                   (int)(uint32_t)(w1 >> 32)};
    if (dev)
        __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, CPOL_SC1);
    else
        __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
}
__device__ __forceinline__ uint32_t stale(uint64_t w, uint32_t tag) { return tag_of(w) ^ tag; }
__device__ __forceinline__ uint32_t stale(const W2 &w, uint32_t tag) {
    return (tag_of(w.a) ^ tag) | (tag_of(w.b) ^ tag);
}

// Order LDS traffic between the lanes of one wave (no workgroup barrier).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- fp32 products on bf16 MFMA ----------------------------------------------
typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef short s4v __attribute__((ext_vector_type(4)));

// bf16 roundings (to nearest even) of a and b, packed (a in the low half)
__device__ __forceinline__ uint32_t bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{a, b}, bf2v));
}
__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Three bf16 parts of a pair: a = a0 + a1 + a2, b likewise; part i of both in
// one word (a in the low half). Each difference below is exact in fp32.
struct Split3 {
    uint32_t p[3];
};
__device__ __forceinline__ Split3 split3(float a, float b) {
    Split3 r;
    r.p[0] = bf16x2(a, b);
    a -= lo_f(r.p[0]);
    b -= hi_f(r.p[0]);
    r.p[1] = bf16x2(a, b);
    a -= lo_f(r.p[1]);
    b -= hi_f(r.p[1]);
    r.p[2] = bf16x2(a, b);
    return r;
}

__device__ __forceinline__ f4 mfma_k32(u4v a, u4v b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8v, a),
                                                   __builtin_bit_cast(bf8v, b), c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfma_k16(u2v a, u2v b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s4v, a),
                                                     __builtin_bit_cast(s4v, b), c, 0, 0, 0);
}
// c += A B with both operands in three parts: the products of part orders
// i + j <= 2, the smallest first
template <class V, class F>
__device__ __forceinline__ f4 mfma3(const V (&a)[3], const V (&b)[3], f4 c, F mfma) {
    c = mfma(a[2], b[0], c);
    c = mfma(a[1], b[1], c);
    c = mfma(a[0], b[2], c);
    c = mfma(a[1], b[0], c);
    c = mfma(a[0], b[1], c);
    return mfma(a[0], b[0], c);
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

// Waits of one wave. A wait that outlives the limit raises the kernel-wide
// abort word and the workgroup's abort stamp (step + 1, in LDS); every later
// wait of the step returns at once, and all waves leave the step loop together
// at the top of the next step.
struct Waiter {
    int *stamp;
    int step;
    bool aborted;

    // Every lane of a wave takes the same branches here: the abort word is read
    // as one wave-uniform value and the deadline comes from the scalar clock.
    __device__ __forceinline__ void check(uint64_t deadline) {
        int32_t *abort = COLD(abort);
        const int ab = __builtin_amdgcn_readfirstlane(
            __hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        if (ab) {
            aborted = true;
        } else if (now_ticks() > deadline) {
            __hip_atomic_store(COLD(err), (int32_t)MLP_ERR_TIMEOUT_CODE, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            aborted = true;
        }
        if (aborted) *stamp = step + 1;
    }
    // w[i] holds a loaded word (or word pair); reload(i) loads it again. Wait
    // until every tag of every lane is current: the test is a wave-wide ballot,
    // so the loop is uniform (no per-lane exits and exec-mask bookkeeping; all
    // lanes reload until the last word has landed, measured 1.5 % faster per
    // step than a divergent loop). With D = 2 two polls are in flight: the next
    // one is issued before the previous is checked, so a word that lands just
    // after a poll left is seen half a round trip sooner. Exchanges B and C
    // (inside an XCD) gain from it; exchange A, whose loads cross XCDs, and
    // deeper pipelines lose (measured: 32-256-1 at batch 4096, 5.24 -> 4.96 us
    // per step with B and C at D = 2; three or four polls in flight, 8.9 us).
    template <int D, int N, class T, class Reload>
    __device__ __forceinline__ void settle(T (&w)[N], uint32_t tag, Reload reload) {
        static_assert(D == 1 || D == 2, "polls in flight");
        auto ok = [&](const T (&x)[N]) {
            uint32_t bad = 0;
#pragma unroll
            for (int i = 0; i < N; ++i) bad |= stale(x[i], tag);
            return __builtin_amdgcn_ballot_w64(bad != 0) == 0;
        };
        if (ok(w) || aborted) return;
        const uint64_t deadline = now_ticks() + COLD(timeout_ticks);
        uint32_t spins = 0;
        if constexpr (D == 1) {
            while (true) {
                asm volatile("" ::: "memory");   // the reloads are not the loads above
#pragma unroll
                for (int i = 0; i < N; ++i) w[i] = reload(i);
                if (ok(w)) break;
                if ((++spins & 63u) == 0) {
                    check(deadline);
                    if (aborted) break;
                }
            }
        } else {
            T v[N];
            asm volatile("" ::: "memory");
#pragma unroll
            for (int i = 0; i < N; ++i) v[i] = reload(i);
            while (true) {
                // w is reissued, then v (the older poll) checked, and the reverse
                asm volatile("" ::: "memory");
#pragma unroll
                for (int i = 0; i < N; ++i) w[i] = reload(i);
                if (ok(v)) {
#pragma unroll
                    for (int i = 0; i < N; ++i) w[i] = v[i];
                    break;
                }
                asm volatile("" ::: "memory");
#pragma unroll
                for (int i = 0; i < N; ++i) v[i] = reload(i);
                if (ok(w)) break;
                if ((++spins & 31u) == 0) {
                    check(deadline);
                    if (aborted) break;
                }
            }
        }
    }
};

// N word pairs per thread of the all-gathered W1 slice (pair i = i0 + 256 q at
// byte offset base + 16 i): its two words carry part p = i / (8 U) of inputs
// 4 m .. 4 m + 3 (m = i % 8) of unit (i / 8) % U, as bf16 pairs, and go to LDS
// in one 8-byte store.
template <int N, int U, int WPS>
__device__ __forceinline__ void gather_parts(Waiter &wt, rsrc_t r, uint32_t base, int i0,
                                             uint32_t tag, uint16_t *WP) {
    W2 w[N];
    auto reload = [&](int q) { return ld2(r, base + 16u * (uint32_t)(i0 + 256 * q)); };
#pragma unroll
    for (int q = 0; q < N; ++q) w[q] = reload(q);
    wt.settle<2>(w, tag, reload);
#pragma unroll
    for (int q = 0; q < N; ++q) {
        const int i = i0 + 256 * q;
        const int p = i / (8 * U), ul = (i / 8) % U, m = i % 8;
        *reinterpret_cast<u2v *>(WP + (p * U + ul) * WPS + 4 * m) =
            u2v{(uint32_t)w[q].a, (uint32_t)w[q].b};
    }
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

// Optional phase accounting (MLP_TRACE=1): compute wave 0 and the first owner
// wave of every workgroup read the core clock (s_memtime) at the boundaries of
// the step's phases, and sum each phase's cycles over the steps from
// PHASE_FROM on; at the end they write, per workgroup and wave, 16 words:
//   [0] steps summed, [1..12] cycles of the phases below, [13] elapsed
//   s_memrealtime ticks (100 MHz) and [14] elapsed core cycles over the summed
//   steps (their ratio is the clock), [15] 0.
// Phases: 1 forward operands from LDS (waited for), 2 forward MFMAs, epilogue
// and exchange-A stores, 3 exchange-A wait of row tile 0, 4 residual of tile 0
// and exchange-A wait of tile 1, 5 residual of the last tile, the backward and
// the P partials into LDS, 6 P barrier, 7 exchange-B stores, 8 exchange-B wait
// (owners), 9 update and exchange-C stores (owners), 10 owners barrier,
// 11 exchange-C gather, 12 step barrier. A phase a wave does not run counts 0.
constexpr int PHASE_FROM = 8, PHASE_WORDS = 16;
#define PHASE(i)                                                                   \
    do {                                                                           \
        if constexpr (TR) {                                                        \
            __builtin_amdgcn_sched_barrier(0);                                     \
            ct[i] = __builtin_amdgcn_s_memtime();                                  \
            __builtin_amdgcn_sched_barrier(0);                                     \
        }                                                                          \
    } while (0)

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
// Compute wave w = wr + wu * WR takes row tiles [wr * RTW, (wr + 1) * RTW) and
// unit tiles {wu + i * WU}. Waves NCW.. are the loaders. Both kinds of wave pass the
// same workgroup barriers: one before the loop, then per step [one more when
// WU > 1,] "P partials ready", [when some compute waves own no units, in training
// mode: "owners done",] and "next step ready".
template <class S, bool TR>
__global__ __launch_bounds__(NTHR) void k_train(const TrainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int s_flags[8];   // 0: group x, 1: rank b, 2: plain local stores, 3: abort stamp, 4: active,
                                 // 5: forward-done stamp (step + 1) of wave 0

    constexpr int R = S::R, U = S::U, PR = S::PR, PX = S::PX, H = S::H;
    constexpr int WR = S::WR, WU = S::WU, NUW = S::NUW, RTW = S::RTW, NRW = S::NRW;
    constexpr int UPW = S::UPW, NPAIR = S::NPAIR, XRS = S::XRS, WPS = S::WPS;
    constexpr int PS = S::PS;
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
    if (tid == 0) {
        s_flags[3] = 0;   // from here on: the abort stamp
        s_flags[5] = 0;
    }

    char *ldsb = reinterpret_cast<char *>(lds);
    uint16_t *XRall = reinterpret_cast<uint16_t *>(ldsb + S::B_XR);   // [2][3][R][XRS]
    uint16_t *WP = reinterpret_cast<uint16_t *>(ldsb + S::B_WP);      // [3][U][WPS]
    float *W2s = reinterpret_cast<float *>(ldsb + S::B_W2);           // [U]
    float *Yall = reinterpret_cast<float *>(ldsb + S::B_Y);           // [2][R]
    float *Ypart = reinterpret_cast<float *>(ldsb + S::B_YP);         // [WU][R]
    float *Pred = reinterpret_cast<float *>(ldsb + S::B_P);           // [WR][U][PS]
    float *SseW = reinterpret_cast<float *>(ldsb + S::B_SSE);         // [NCW]
    // a weight-slice value into LDS: W1 (k < 32) in three bf16 parts, W2 as is
    auto put_w = [&](int j, int k, float v) {
        if (k < 32) {
            const Split3 q = split3(v, 0.0f);
#pragma unroll
            for (int p = 0; p < 3; ++p) WP[(p * U + j) * WPS + k] = (uint16_t)q.p[p];
        } else {
            W2s[j] = v;
        }
    };

    const int steps = (int)a.steps;
    const int spe = (int)((a.n + a.batch - 1) / a.batch);
    const int batch = (int)a.batch;
    const int tail = (int)(a.n - (int64_t)(spe - 1) * a.batch);

    if (run) {
        // ---- the group's weight slice (all waves) ---------------------------------
        for (int i = tid; i < U * 33; i += NTHR) {
            const int jl = i / 33, k = i - jl * 33;
            const int ug = gx * U + jl;
            put_w(jl, k, k < 32 ? COLD(W1)[k * H + ug] : COLD(W2)[ug]);
        }
        Waiter wt{&s_flags[3], 0, false};

        if (wave < NCW) {
            // ================= compute waves =================================
            // exchange buffers: A [2][PR][PX][RMAX], B [2][PX][GBW], C [2][PX][CW] words
            const rsrc_t rA = make_rsrc(a.xch, 8u * (uint32_t)(2 * PR * PX * RMAX));
            const rsrc_t rB = make_rsrc(a.rs, 8u * (uint32_t)(2 * PX * S::GBW));
            const rsrc_t rC = make_rsrc(a.ag, 8u * (uint32_t)(2 * PX * S::CW));
            const int wr = wave % WR, wu = wave / WR;
            constexpr int KPW = S::KPW, SG = S::SG, LPS = S::LPS;
            // the owner waves are the last NWO compute waves (the loader shares SIMD 0
            // with wave 0)
            constexpr int OW0 = NCW - S::NWO;
            const bool owner = wave >= OW0;
            const int kp = (wave - OW0) * KPW + lane % KPW;     // owned k pair
            const int sg = lane / KPW;                          // source group
            const int jl = kp >> 4, k0 = 2 * (kp & 15);         // owned unit, first k of the pair
            const int ug = gx * U + gb * UPW + jl;
            float ow1a = 0.f, ow1b = 0.f, ow2 = 0.f;            // master copy of the owned words
            if (owner) {
                ow1a = COLD(W1)[k0 * H + ug];
                ow1b = COLD(W1)[(k0 + 1) * H + ug];
                ow2 = COLD(W2)[ug];
            }
            float scale_full = 2.0f / (float)batch, scale_tail = 2.0f / (float)tail;
            asm volatile("" : "+v"(scale_full), "+v"(scale_tail));   // computed once, selected per step
            // the loss is reduced one step late by wave 1 of workgroup (0, 0)
            const bool lossw = gx == 0 && gb == 0 && wave == 1;
            double epoch_sse = 0.0;
            uint64_t ct[13] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};   // phase stamps
            uint64_t cacc[PHASE_WORDS] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
            uint64_t rt0 = 0, mt0 = 0;
            Pos cur{0, 0}, prev{0, 0};
            int nb_prev = 1;
            int done = 0;
            __syncthreads();                                    // weights and the first rows staged

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
                const float scale = cur.sb == spe - 1 ? scale_tail : scale_full;   // 2 / nb
                const uint16_t *XRb = XRall + par * 3 * R * XRS;
                const float *Yb = Yall + par * R;
                const uint32_t bB = 8u * (uint32_t)((par * PX + gx) * S::GBW);   // group block (bytes)
                PHASE(0);
                if constexpr (TR)
                    if (s == PHASE_FROM) {
                        rt0 = now_ticks();
                        mt0 = ct[0];
                    }

                // deferred loss: issue the loads of the previous step's SSE partials
                const uint32_t tag_prev = tag - 1;
                const uint32_t sse_prev = 8u * (uint32_t)(((par ^ 1) * PX) * S::GBW + PR * S::RSW +
                                                          (lane < PR ? lane : 0));
                uint64_t sw[1] = {pack(0.f, tag_prev)};
                if (lossw && s > 0 && lane < PR) sw[0] = ld1(rB, sse_prev);

                // ---- 1. forward: Z1 tiles, mask bits, partial Ypred ---------------
                // With one unit wave per row block (WU == 1) the row sums go straight
                // to exchange A, tile by tile; otherwise they meet in LDS first.
                constexpr bool DIRECT = WU == 1 && PX > 1;
                const uint32_t bA = 8u * (uint32_t)((par * PR + gb) * PX * RMAX);
                // B operand (read at each use, to bound registers): W1 inputs
                // 8 lq .. 8 lq + 7 of unit li of unit tile u
                auto wpart = [&](int u, int p) {
                    return *reinterpret_cast<const u4v *>(WP + (p * U + (wu + u * WU) * 16 + li) * WPS + 8 * lq);
                };
                float w2v[NUW];
#pragma unroll
                for (int u = 0; u < NUW; ++u) w2v[u] = W2s[(wu + u * WU) * 16 + li];
                if constexpr (TR) {
                    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the weight operands
                    PHASE(1);
                }
                uint32_t mbits = 0;   // bit (i*NUW + u)*4 + v
#pragma unroll
                for (int i = 0; i < RTW; ++i) {
                    const int tile = wr * RTW + i;
                    // A operand: row li of the tile, inputs 8 lq .. 8 lq + 7
                    u4v xq[3];
#pragma unroll
                    for (int p = 0; p < 3; ++p)
                        xq[p] = *reinterpret_cast<const u4v *>(XRb + (p * R + tile * 16 + li) * XRS + 8 * lq);
                    // the target group 0 folds into its exchange-A word, read ahead of
                    // the MFMAs so that the store does not wait on LDS
                    const float yv = (DIRECT && gx == 0) ? Yb[tile * 16 + 4 * lq + (li >> 2)] : 0.0f;
                    f4 acc[NUW];
#pragma unroll
                    for (int u = 0; u < NUW; ++u) {
                        const u4v wq[3] = {wpart(u, 0), wpart(u, 1), wpart(u, 2)};
                        acc[u] = mfma3(xq, wq, f4{0.f, 0.f, 0.f, 0.f}, mfma_k32);
                    }
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
                    // lane li of row group g gets the sum of row 4 g + (li >> 2)
                    const float rowv = rsum16x4(yp, li);
                    if constexpr (DIRECT) {
                        // lanes li = 4 v store row 4 g + v, so the tile's 16 words go
                        // out in one store; group 0 folds -Y into its partial, so the
                        // group sum is the residual Ypred - Y and the other groups
                        // need no targets
                        if ((li & 3) == 0) {
                            const int row = tile * 16 + 4 * lq + (li >> 2);
                            st1(rA, bA + 8u * (uint32_t)(gx * RMAX + row), pack(rowv - yv, tag), true);
                        }
                    } else {
                        if ((li & 3) == 0) Ypart[wu * R + tile * 16 + 4 * lq + (li >> 2)] = rowv;
                    }
                }
                if (wave == 0 && lane == 0) s_flags[5] = s + 1;   // the loader may start
                if constexpr (WU > 1)
                    __syncthreads();   // partial Ypred of the unit waves
                else
                    wave_sync();
                if constexpr (!DIRECT && PX > 1) {
                    if (wu == 0 && lane < NRW) {
                        float v = 0.f;
#pragma unroll
                        for (int w = 0; w < WU; ++w) v += Ypart[w * R + wr * NRW + lane];
                        if (gx == 0) v -= Yb[wr * NRW + lane];   // residual, as above
                        st1(rA, bA + 8u * (uint32_t)(gx * RMAX + wr * NRW + lane), pack(v, tag), true);
                    }
                }
                asm volatile("" ::: "memory");
                PHASE(2);

                // ---- 2. exchange A, residual and backward, one row tile at a time --
                // lane (lq, li): rows 4 lq + 2 h, 4 lq + 2 h + 1 (h = li >> 3) of the
                // tile from group peer li & 7; the group sums run as a symmetric
                // butterfly over the 8 lanes of a half-row (a fixed order), and the
                // other half-row supplies the lane's other two rows, so each lane
                // ends with dZ2 of exactly the rows its backward MFMA operands need.
                // The backward of a tile overlaps the exchange of the next.
                const int hh = li >> 3;
                const int peer = (li & 7) % PX;
                W2 wa[RTW];
                if constexpr (PX > 1) {
#pragma unroll
                    for (int i = 0; i < RTW; ++i)
                        wa[i] = ld2(rA, bA + 8u * (uint32_t)(peer * RMAX + (wr * RTW + i) * 16 + 4 * lq + 2 * hh));
                }
                // the backward's A operands (input kt * 16 + li; rows 4 lq .. 4 lq + 3
                // of each of the wave's row tiles, 16-bit reads) come out of LDS
                // while exchange A is in flight
                u2v xtq[2][3][RTW];
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int p = 0; p < 3; ++p)
#pragma unroll
                        for (int i = 0; i < RTW; ++i) {
                            const uint16_t *xp = XRb + (p * R + (wr * RTW + i) * 16 + 4 * lq) * XRS + kt * 16 + li;
                            xtq[kt][p][i] = u2v{(uint32_t)xp[0] | ((uint32_t)xp[XRS] << 16),
                                                (uint32_t)xp[2 * XRS] | ((uint32_t)xp[3 * XRS] << 16)};
                        }
                // deferred loss of the previous step, reduced while exchange A is in
                // flight: its words are long written, and they stay intact at least
                // until this workgroup has passed the barrier below (no group-0
                // workgroup can store the next step's words before every owner of
                // group 0 has this workgroup's exchange-B words)
                if (lossw && s > 0) {
                    wt.settle<1>(sw, tag_prev, [&](int) { return lane < PR ? ld1(rB, sse_prev) : pack(0.f, tag_prev); });
                    const float sse = sum64(lane < PR ? val_of(sw[0]) : 0.0f);
                    if (lane == 0) {
                        flag_nonfinite(sse, COLD(err));
                        const float L = sse / (float)nb_prev;               // eq. 14
                        float *lo = COLD(loss), *sl = COLD(step_loss), *el = COLD(epoch_loss);
                        if (lo) lo[0] = L;
                        if (sl) sl[s - 1] = L;
                        if (prev.sb == 0) epoch_sse = 0.0;
                        epoch_sse += (double)sse;
                        if (el) el[prev.e] = (float)(epoch_sse * (double)COLD(inv_n));
                    }
                }
                float r2acc = 0.f;
                Split3 gq[RTW][2];   // dZ2 of rows 4 lq + v of each row tile, in parts (v = 0,1 | 2,3)
#pragma unroll
                for (int i = 0; i < RTW; ++i) {
                    const int tile = wr * RTW + i;
                    const int ra = tile * 16 + 4 * lq + 2 * hh;   // first row of the lane's pair
                    float y0 = 0.f, y1 = 0.f;
                    if constexpr (PX > 1) {
                        W2 one[1] = {wa[i]};
                        wt.settle<1>(one, tag, [&](int) {
                            return ld2(rA, bA + 8u * (uint32_t)(peer * RMAX + ra));
                        });
                        y0 = val_of(one[0].a);
                        y1 = val_of(one[0].b);
                        if (i == 0) PHASE(3); else PHASE(4);
                        if constexpr (PX == 8) {
                            y0 += dppf<0x141>(y0);   // row_half_mirror: lanes i, 7 - i
                            y1 += dppf<0x141>(y1);
                        }
                        if constexpr (PX >= 4) {
                            y0 += dppf<0x4E>(y0);    // lanes i, i ^ 2
                            y1 += dppf<0x4E>(y1);
                        }
                        y0 += dppf<0xB1>(y0);        // lanes i, i ^ 1
                        y1 += dppf<0xB1>(y1);
                    } else {
#pragma unroll
                        for (int w = 0; w < WU; ++w) {
                            y0 += Ypart[w * R + ra];
                            y1 += Ypart[w * R + ra + 1];
                        }
                    }
                    // residual, dZ2 (eqs. 14-15), squared residuals
                    float gv[4];
                    {
                        // across groups the exchanged sum is already Ypred - Y
                        const float e0 = PX > 1 ? y0 : y0 - Yb[ra], e1 = PX > 1 ? y1 : y1 - Yb[ra + 1];
                        const bool in0 = ra < rc, in1 = ra + 1 < rc;
                        const float g0 = in0 ? scale * e0 : 0.0f, g1 = in1 ? scale * e1 : 0.0f;
                        if ((li & 7) == 0 && wu == 0) r2acc += (in0 ? e0 * e0 : 0.0f) + (in1 ? e1 * e1 : 0.0f);
                        const float o0 = dppf<0x128>(g0), o1 = dppf<0x128>(g1);   // lane li ^ 8
                        gv[0] = hh ? o0 : g0;
                        gv[1] = hh ? o1 : g1;
                        gv[2] = hh ? g0 : o0;
                        gv[3] = hh ? g1 : o1;
                    }
                    gq[i][0] = split3(gv[0], gv[1]);
                    gq[i][1] = split3(gv[2], gv[3]);
                }
                // ---- 3. backward: P += X^T (dZ2 (.) mask) over the wave's rows ------
                // K index 8 lq + j (4 lq + j with one row tile): row 4 lq + (j & 3) of
                // row tile j >> 2, so that both operands hold only the lane's own rows
                f4 pacc[2][NUW];
#pragma unroll
                for (int u = 0; u < NUW; ++u) {
                    // B operand: dZ2 (.) ReLU'(Z1) of the unit li, in parts
                    uint32_t bm[RTW][2][3];
#pragma unroll
                    for (int i = 0; i < RTW; ++i)
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const uint32_t bits = mbits >> ((i * NUW + u) * 4 + 2 * h);
                            const uint32_t keep = ((bits & 1u) ? 0x0000FFFFu : 0u) | ((bits & 2u) ? 0xFFFF0000u : 0u);
#pragma unroll
                            for (int p = 0; p < 3; ++p) bm[i][h][p] = gq[i][h].p[p] & keep;
                        }
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) {
                        if constexpr (RTW == 2) {
                            u4v aq[3], bq[3];
#pragma unroll
                            for (int p = 0; p < 3; ++p) {
                                aq[p] = u4v{xtq[kt][p][0].x, xtq[kt][p][0].y, xtq[kt][p][1].x, xtq[kt][p][1].y};
                                bq[p] = u4v{bm[0][0][p], bm[0][1][p], bm[1][0][p], bm[1][1][p]};
                            }
                            pacc[kt][u] = mfma3(aq, bq, f4{0.f, 0.f, 0.f, 0.f}, mfma_k32);
                        } else {
                            u2v aq[3], bq[3];
#pragma unroll
                            for (int p = 0; p < 3; ++p) {
                                aq[p] = xtq[kt][p][0];
                                bq[p] = u2v{bm[0][0][p], bm[0][1][p]};
                            }
                            pacc[kt][u] = mfma3(aq, bq, f4{0.f, 0.f, 0.f, 0.f}, mfma_k16);
                        }
                    }
                }
                {
                    const float sse = sum64(r2acc);
                    if (lane == 0) SseW[wave] = sse;
                }
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int u = 0; u < NUW; ++u) {
                        // the lane's four k = kt * 16 + 4 lq + v of unit ul, in one store
                        const int ul = (wu + u * WU) * 16 + li;
                        *reinterpret_cast<float4 *>(Pred + (wr * U + ul) * PS + kt * 16 + 4 * lq) =
                            make_float4(pacc[kt][u][0], pacc[kt][u][1], pacc[kt][u][2], pacc[kt][u][3]);
                    }

                if constexpr (TR) {
                    if constexpr (PX == 1) {   // no exchange A: both of its waits count 0
                        ct[3] = ct[2];
                        ct[4] = ct[2];
                    } else if constexpr (RTW == 1) {
                        ct[4] = ct[3];
                    }
                }
                PHASE(5);
                __syncthreads();   // P partials and SSE of every wave in LDS
                PHASE(6);

                // ---- 4. exchange B: reduce-scatter of P inside the group ---------
                // word (ul, k) of this workgroup goes to owner o = ul / UPW at word
                // (o * PR + gb) * NPAIR + (ul % UPW) * 32 + k of the group block
                {
                    // every LDS operand of this workgroup's exchange-B words first (one
                    // LDS round trip), then the sums and the stores
                    constexpr int NIT = S::RSW / 512;
                    float2 pv[NIT][WR];
                    float sv[WR];
#pragma unroll
                    for (int it = 0; it < NIT; ++it) {
                        const int i = it * 512 + 2 * tid;
                        const int ul = i >> 5, k = i & 31;
#pragma unroll
                        for (int w = 0; w < WR; ++w)
                            pv[it][w] = *reinterpret_cast<const float2 *>(Pred + (w * U + ul) * PS + k);
                    }
#pragma unroll
                    for (int w = 0; w < WR; ++w) sv[w] = SseW[w];
#pragma unroll
                    for (int it = 0; it < NIT; ++it) {
                        const int i = it * 512 + 2 * tid;
                        const int ul = i >> 5, k = i & 31;
                        float v0 = 0.f, v1 = 0.f;
#pragma unroll
                        for (int w = 0; w < WR; ++w) {
                            v0 += pv[it][w].x;
                            v1 += pv[it][w].y;
                        }
                        const int o = ul / UPW, jo = ul - o * UPW;
                        st2(rB, bB + 8u * (uint32_t)((o * PR + gb) * NPAIR + jo * 32 + k), pack(v0, tag),
                            pack(v1, tag), !plain);
                    }
                    if (tid == 0) {
                        float v = 0.f;
#pragma unroll
                        for (int w = 0; w < WR; ++w) v += sv[w];
                        st1(rB, bB + 8u * (uint32_t)(PR * S::RSW + gb), pack(gx == 0 ? v : 0.f, tag), !plain);
                    }
                }
                asm volatile("" ::: "memory");
                PHASE(7);
                ct[8] = ct[7];
                ct[9] = ct[7];
                if (owner) {
                    // words (k0, k0 + 1) of unit jl from sources sg * LPS + b, in source order
                    // (in chunks of at most 8 sources, to bound registers)
                    constexpr int CHB = LPS < 8 ? LPS : 8;
                    static_assert(LPS % CHB == 0, "owner chunks");
                    float p0 = 0.f, p1 = 0.f;
#pragma unroll
                    for (int c = 0; c < LPS / CHB; ++c) {
                        const uint32_t ob =
                            bB + 8u * (uint32_t)((gb * PR + sg * LPS + c * CHB) * NPAIR + 2 * kp);
                        W2 w[CHB];
                        auto reload = [&](int b) { return ld2(rB, ob + 8u * (uint32_t)(b * NPAIR)); };
#pragma unroll
                        for (int b = 0; b < CHB; ++b) w[b] = reload(b);
                        wt.settle<2>(w, tag, reload);
#pragma unroll
                        for (int b = 0; b < CHB; ++b) {
                            p0 += val_of(w[b].a);
                            p1 += val_of(w[b].b);
                        }
                    }
                    if constexpr (SG == 4) {   // lane groups of 16
                        p0 = xadd32(xadd16(p0));
                        p1 = xadd32(xadd16(p1));
                    } else if constexpr (SG == 2) {   // lane groups of 32
                        p0 = xadd32(p0);
                        p1 = xadd32(p1);
                    }
                    PHASE(8);
                    // ---- update the owned units (eq. 19) or emit gradients ------
                    const float dw1a = ow2 * p0, dw1b = ow2 * p1;       // dW1_kj = W2_j P_kj
                    const float dw2 = rsum16(fmaf(ow1b, p1, ow1a * p0)); // dW2_j = sum_k W1_kj P_kj
                    if (a.mode == 1) {
                        if (sg == 0) {
                            float *dW1 = COLD(dW1);
                            dW1[k0 * H + ug] = dw1a;
                            dW1[(k0 + 1) * H + ug] = dw1b;
                            if (k0 == 0) COLD(dW2)[ug] = dw2;
                        }
                    } else {
                        ow1a -= a.lr * dw1a;
                        ow1b -= a.lr * dw1b;
                        ow2 -= a.lr * dw2;
                        if (sg == 0) {
                            // the pair (k0, k0 + 1) in three bf16 parts, one word each, and W2
                            const uint32_t cb = 8u * (uint32_t)((par * PX + gx) * S::CW);
                            const int ul = gb * UPW + jl;
                            const Split3 q = split3(ow1a, ow1b);
#pragma unroll
                            for (int p = 0; p < 3; ++p)
                                st1(rC, cb + 8u * (uint32_t)((p * U + ul) * 16 + (k0 >> 1)),
                                    pack(__uint_as_float(q.p[p]), tag), !plain);
                            if (k0 == 0) st1(rC, cb + 8u * (uint32_t)(48 * U + ul), pack(ow2, tag), !plain);
                        }
                    }
                    PHASE(9);
                }
                asm volatile("" ::: "memory");

                // ---- 5. exchange C: all-gather the group's updated slice ---------
                // the other waves start polling once this workgroup's owners are
                // done: the group's words are then about to land, and earlier
                // polls would only load the L2 while exchange B is under way
                if constexpr (S::NWO < NCW)
                    if (a.mode == 0) __syncthreads();
                PHASE(10);
                if (a.mode == 0) {
                    // the W1 parts in chunks of CHC word pairs per thread (to bound
                    // registers); the W2 words (threads below U / 2) load first
                    const uint32_t cbase = 8u * (uint32_t)((par * PX + gx) * S::CW);
                    W2 wr1[1] = {W2{pack(0.f, tag), pack(0.f, tag)}};
                    auto reload1 = [&](int) {
                        return tid < U / 2 ? ld2(rC, cbase + 8u * (uint32_t)(48 * U + 2 * tid))
                                           : W2{pack(0.f, tag), pack(0.f, tag)};
                    };
                    wr1[0] = reload1(0);
#pragma unroll
                    for (int c = 0; c < S::NPW / S::CHC; ++c)
                        gather_parts<S::CHC, U, WPS>(wt, rC, cbase, tid + 256 * S::CHC * c, tag, WP);
                    wt.settle<2>(wr1, tag, reload1);
                    if (tid < U / 2) {
                        W2s[2 * tid] = val_of(wr1[0].a);
                        W2s[2 * tid + 1] = val_of(wr1[0].b);
                    }
                }
                PHASE(11);
                prev = cur;
                nb_prev = nb;
                cur.advance(spe);
                done = s + 1;
                __syncthreads();   // next step's rows staged, weight slice updated
                PHASE(12);
                if constexpr (TR)
                    if (s >= PHASE_FROM) {
#pragma unroll
                        for (int q = 1; q < 13; ++q) cacc[q] += ct[q] - ct[q - 1];
                        cacc[0] += 1;
                        cacc[13] = now_ticks() - rt0;
                        cacc[14] = ct[12] - mt0;
                    }
            }
            if constexpr (TR)
                if (a.phase && lane == 0) {
                    // slot 0: compute wave 0; slot 1: the first owner wave (the same
                    // wave when every compute wave owns units)
#pragma unroll
                    for (int sl = 0; sl < 2; ++sl)
                        if (wave == (sl == 0 ? 0 : OW0))
#pragma unroll
                            for (int q = 0; q < PHASE_WORDS; ++q)
                                a.phase[((gx * S::PR + gb) * 2 + sl) * PHASE_WORDS + q] = cacc[q];
                }

            // ---- after the loop -----------------------------------------------------
            const bool aborted = s_flags[3] != 0;
            if (!aborted && done > 0 && lossw) {
                // loss of the last step
                const uint32_t tag_last = a.tag_base + (uint32_t)(done - 1);
                const uint32_t sse_last = 8u * (uint32_t)((((done - 1) & 1) * PX) * S::GBW + PR * S::RSW +
                                                          (lane < PR ? lane : 0));
                auto reload = [&](int) { return lane < PR ? ld1(rB, sse_last) : pack(0.f, tag_last); };
                uint64_t swl[1] = {reload(0)};
                wt.settle<1>(swl, tag_last, reload);
                const float sse = sum64(lane < PR ? val_of(swl[0]) : 0.0f);
                if (lane == 0) {
                    flag_nonfinite(sse, COLD(err));
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
            if (a.mode == 0 && owner && sg == 0) {
                float *W1 = COLD(W1);
                W1[k0 * H + ug] = ow1a;
                W1[(k0 + 1) * H + ug] = ow1b;
                if (k0 == 0) COLD(W2)[ug] = ow2;
            }
        } else {
            // ================= loader waves ===================================
            // loader wave l takes rows {8 l + r8 + 16 j}
            // Indices are loaded two steps ahead and rows one step ahead into
            // registers; a step's rows are written to LDS during the step before.
            constexpr int RPL = S::RPL;
            const int lc = lane & 7, lr0 = (lane >> 3) + 8 * (wave - NCW);   // float4 chunk, first row
            const int64_t row0 = (int64_t)gb * R;
            const bool needy = PX == 1 || gx == 0;   // only group 0 uses the targets
            int32_t pidx[RPL];
            float4 pfx[RPL];
            float pfy[RPL];
            // indices of a step: one load, lane m (m < R/2) holding row
            // 8 l + m % 8 + 16 (m / 8) of loader wave l; spread to the row lanes
            // when the rows are fetched
            int32_t cidx = 0;
            auto fetch_idx = [&](const Pos &ps) {
                const int64_t off = (int64_t)ps.sb * COLD(batch);
                const int32_t *perm = COLD(perm);
                const int64_t n = COLD(n);
                const int m = lane < R / 2 ? lane : 0;
                const int64_t pos = off + row0 + 8 * (wave - NCW) + (m & 7) + 16 * (m >> 3);
                if (perm)
                    cidx = perm[(int64_t)ps.e * n + (pos < n ? pos : n - 1)];   // always a valid address
                else
                    cidx = (int32_t)pos;
            };
            auto fetch_rows = [&](const Pos &ps) {
#pragma unroll
                for (int j = 0; j < RPL; ++j) pidx[j] = __shfl(cidx, 8 * j + (lane >> 3), 64);
                const int nbr = ps.sb == spe - 1 ? tail : batch;
                const int64_t rcl = nbr - row0;
                const float *X = COLD(X), *Y = COLD(Y);
                const int64_t n_rows = COLD(n_rows);
#pragma unroll
                for (int j = 0; j < RPL; ++j) {
                    const int r = lr0 + 8 * NLW * j;
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
                        if (lc == 0 && needy) y = Y[row];
                    }
                    pfx[j] = v;
                    pfy[j] = y;
                }
            };
            // a row's inputs 4 lc .. 4 lc + 3 in three bf16 parts
            auto stage = [&](int buf) {
                uint16_t *XRd = XRall + buf * 3 * R * XRS;
                float *Yd = Yall + buf * R;
#pragma unroll
                for (int j = 0; j < RPL; ++j) {
                    const int r = lr0 + 8 * NLW * j;
                    const Split3 s01 = split3(pfx[j].x, pfx[j].y), s23 = split3(pfx[j].z, pfx[j].w);
#pragma unroll
                    for (int p = 0; p < 3; ++p)
                        *reinterpret_cast<u2v *>(XRd + (p * R + r) * XRS + 4 * lc) = u2v{s01.p[p], s23.p[p]};
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
                // wait until wave 0 has finished its forward pass: the compute waves
                // then wait on exchange A, and the loader's work stays off their path
                {
                    const volatile int *fd = &s_flags[5];
                    while (*fd < s + 1) __builtin_amdgcn_s_sleep(1);
                }
                // registers hold the rows of step s+1 and the indices of step s+2
                // (position q2)
                if (s + 1 < steps) stage((s + 1) & 1);
                Pos q3 = q2;
                q3.advance(spe);
                if (s + 2 < steps) fetch_rows(q2);
                if (s + 3 < steps) fetch_idx(q3);
                q2 = q3;
                __syncthreads();   // P partials ready
                if constexpr (S::NWO < NCW)
                    if (a.mode == 0) __syncthreads();   // owners done
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

// The kernel needs every workgroup resident at once (its waits span the grid).
// A cooperative launch guarantees that. With regular = true (a diagnostic hook
// for profiler runs, MLP_REGULAR_LAUNCH=1) the same kernel is launched
// normally: one workgroup per CU by its LDS request, grid <= CUs, and the
// kernel's start barrier times out with MLP_ERR_TIMEOUT rather than wait
// forever if some workgroup cannot start.
template <class S>
static hipError_t launch_shape(hipStream_t stream, TrainArgs &a, bool regular) {
    void *args[] = {&a};
    const void *fn = a.phase ? reinterpret_cast<const void *>(&k_train<S, true>)
                             : reinterpret_cast<const void *>(&k_train<S, false>);
    if (regular)
        return hipLaunchKernel(fn, dim3(a.plan.grid), dim3(NTHR), args, (size_t)a.plan.lds, stream);
    return hipLaunchCooperativeKernel(fn,
                                      dim3(a.plan.grid), dim3(NTHR), args, (unsigned)a.plan.lds,
                                      stream);
}

// Modelled step time (seconds): MFMA work of one wave (six bf16 MFMAs of about
// 17 cycles at 2.4 GHz per fp32 product tile: forward RTW * NUW tiles, backward
// 2 * NUW), exchange A across XCDs when PX > 1,
// the rounds of exchanges B and C (each round one load round trip) and the
// owner's loads per lane. The constants are fitted to step times measured on
// MI355X (at batch 64 and 256, eight groups of few workgroups beat one group of
// many or four groups).
template <class S>
static double shape_cost() {
    constexpr int CHB = S::LPS < 8 ? S::LPS : 8;
    constexpr int rounds_b = S::LPS / CHB;
    constexpr int rounds_c = S::NPW / S::CHC;
    const double compute = 17.0 * 6.0 * S::NUW * (S::RTW + 2) / 2.4e9;
    return compute + (S::PX > 1 ? 1.5e-6 : 0.0) + 0.6e-6 * rounds_b + 0.05e-6 * S::LPS +
           0.5e-6 * rounds_c;
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
    const size_t bytes = (size_t)S::LDS_BYTES;
    const size_t one_per_cu = 84 * 1024;   // > half of the 160 KB LDS: one workgroup per CU
    p.lds = bytes > one_per_cu ? bytes : one_per_cu;
    p.cost = shape_cost<S>();
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
    X(12, 2, 16, 16, 128)  /* 32-256-1,  batch <= 256, two XCDs */    \
    X(13, 4, 4, 16, 64)    /* 32-256-1,  batch <= 64,  four XCDs */   \
    X(14, 8, 4, 32, 32)    /* 32-256-1,  batch <= 128 */              \
    X(15, 8, 8, 32, 32)    /* 32-256-1,  batch <= 256 */

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

// Test and diagnostic hooks, read from the environment (none skips work):
//   MLP_PX=p, MLP_INST=i   restrict the choice to shapes with PX = p, or to
//                          instance i (the parity tests run every instantiated
//                          shape this way);
//   MLP_FORCE_COHERENT=1   device-coherent exchange stores even when every group
//                          sits on one XCD (tested bitwise against the default);
//   MLP_TRACE=1            per-phase cycle sums of every workgroup into the
//                          workspace (read with mlp_phase_cycles);
//   MLP_REGULAR_LAUNCH=1   a regular launch instead of a cooperative one (the
//                          same kernel and grid; for profiler runs, which end
//                          with SIGSEGV after any cooperative launch).
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
        const double cst = pl.cost;
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
// two parities x (three bf16-part words per W1 pair of inputs, one W2 word) per unit
size_t persist_words_ag(int hidden) { return (size_t)2 * hidden * 49; }

hipError_t launch_train(Ctx &c, TrainArgs &a) {
    a.xch = c.xch;
    a.rs = c.rs;
    a.ag = c.ag;
    a.reg = c.ctl->reg;
    a.abort = &c.ctl->abort;
    a.err = &c.ctl->err;
    a.timeout_ticks = 200000000ull;   // 2 s
    const char *tr = getenv("MLP_TRACE");
    a.phase = (tr && tr[0] == '1') ? reinterpret_cast<uint64_t *>(c.slots) : nullptr;
    c.phase_words = a.phase ? (int64_t)a.plan.grid * 2 * PHASE_WORDS : 0;
    const char *fc = getenv("MLP_FORCE_COHERENT");
    a.force_coherent = (fc && fc[0] == '1') ? 1 : 0;
    // tags of the next call start past every tag this call can use; a range
    // that would leave 32 bits restarts at 1 over cleared exchange words
    const TagPlan tp = plan_tags(c.tag_base, a.steps);
    if (tp.clear) {
        const hipError_t e = clear_words(c, c.xch, c.xch_words);
        if (e != hipSuccess) return e;
    }
    a.tag_base = tp.base;
    c.tag_base = tp.next;
    const char *rl = getenv("MLP_REGULAR_LAUNCH");
    const bool regular = rl && rl[0] == '1' && c.num_cu >= a.plan.grid;
    switch (a.plan.inst) {
#define MLP_SHAPE_CASE(I, PX, PR, R, U) \
    case I: return launch_shape<Shape##I>(c.stream, a, regular);
        MLP_SHAPES(MLP_SHAPE_CASE)
#undef MLP_SHAPE_CASE
    }
    return hipErrorInvalidValue;
}

}  // namespace mlp
