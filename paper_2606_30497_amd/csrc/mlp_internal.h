// mlp_internal.h -- shared declarations of the HIP implementation of mlp.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mlp.h"

struct mlp_ctx;

namespace mlp {

constexpr int D_IN = 32;          // input width (paper Sec. III.A)
constexpr int TILE_SLOTS = 256;   // most workgroups of one tile-path step
constexpr size_t CTL_BYTES = 4096;

constexpr int32_t MLP_ERR_TIMEOUT_CODE = MLP_ERR_TIMEOUT;

// Raise the sticky MLP_ERR_NONFINITE when a batch's sum of squared residuals is
// NaN or infinite (the comparison is false for NaN).
__device__ __forceinline__ void flag_nonfinite(float sse, int32_t *err) {
    if (!(fabsf(sse) <= 3.40282347e38f))
        __hip_atomic_store(err, (int32_t)MLP_ERR_NONFINITE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Control words at the head of the workspace.
struct Control {
    int32_t err;          // sticky kernel-side error (an mlp_status code)
    int32_t abort;        // persistent trainer: set when a wait times out
    double epoch_sse;     // tile path: running sum of squared residuals of the epoch
    int32_t pad0[60];
    int32_t reg[64];      // persistent trainer: registration / start / exit counters
    uint32_t pad[128];
};
static_assert(sizeof(Control) <= CTL_BYTES, "control block too large");

// Launch plan of the persistent trainer (see train_persistent.hip).
struct TrainPlan {
    int inst = -1;      // instantiated shape
    int px = 0;         // groups (one per XCD), each owns U = hidden / px units
    int pr = 0;         // workgroups per group; each takes R rows of a batch
    int R = 0;          // rows per workgroup (multiple of 16, <= RMAX)
    int U = 0;          // units per group (multiple of 16)
    int wr = 1, wu = 4; // waves along rows x waves along units (wr * wu = 4)
    int nuw = 1;        // unit tiles per wave
    int rtw = 1;        // row tiles per wave
    int upw = 1;        // units owned (reduced and updated) per workgroup = U / pr
    int rmax = 0;       // words per workgroup in the exchange-A buffer
    int rs_stride = 0;  // words per workgroup in the exchange-B buffer
    int grid = 0;       // workgroups launched (8 * pr)
    size_t lds = 0;     // dynamic LDS bytes
    double cost = 0.0;  // modelled seconds per step
};

struct TrainArgs {
    const float *X;
    const float *Y;
    int64_t n_rows;           // rows of X and Y
    const int32_t *perm;      // [epochs x n] or null (identity order)
    int64_t n;                // rows visited per epoch
    int64_t batch;
    int64_t steps;            // steps to run in this call
    float lr;
    float inv_n;
    int32_t mode;             // 0: SGD (update weights), 1: gradient only (one step)
    int32_t hidden;
    int32_t epochs;
    float *W1, *W2;           // caller's weights (read at start, written at end)
    float *dW1, *dW2;         // mode 1 outputs
    float *loss;              // nullable [1]
    float *step_loss;         // nullable [steps]
    float *epoch_loss;        // nullable [epochs]
    uint64_t *xch, *rs, *ag;  // exchange buffers
    int32_t *reg;             // registration counters (cleared by the last workgroup)
    int32_t *abort;
    int32_t *err;
    uint32_t tag_base;        // tags of this call: tag_base + step
    uint64_t timeout_ticks;   // per-wait limit in s_memrealtime ticks (100 MHz)
    int32_t force_coherent;   // 1: device-coherent stores even when placement checks out
    uint64_t *phase;          // nullable: per-phase cycle sums of every workgroup
    TrainPlan plan;
};

constexpr int RMAX = 256;         // largest rows per workgroup of the persistent trainer

struct Ctx {
    int hidden = 0;
    int64_t max_batch = 0;
    float *W1 = nullptr;      // caller's [32 x hidden]
    float *W2 = nullptr;      // caller's [hidden]
    Control *ctl = nullptr;   // workspace head
    float *slots = nullptr;   // TILE_SLOTS partial slots
    int64_t slot_stride = 0;  // floats per slot
    uint64_t *xch = nullptr;  // persistent trainer exchange buffers
    uint64_t *rs = nullptr;
    uint64_t *ag = nullptr;
    int64_t xch_words = 0;    // words of the three exchange buffers (cleared to tag 0)
    int64_t phase_words = 0;  // phase-cycle words the last traced trainer call wrote
    uint32_t tag_base = 1;
    hipStream_t stream = nullptr;
    int device = 0;
    int num_cu = 0;
    bool profile = false;
    int strategy = MLP_STRATEGY_FUSED;
    float *hl_ws = nullptr;       // OPTIMIZED / BASELINE intermediates (caller's memory)
    int64_t hl_max_batch = 0;     // batch the strategy workspace was sized for
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    bool ev_valid = false;
};

// Arguments of the slot reduction (tile path).
struct ReduceArgs {
    int sgd;                  // 1: W -= lr dW; 0: write dW1/dW2
    float lr;
    float inv_nb;             // 1 / rows of this batch
    float inv_n;              // 1 / rows of the dataset (epoch loss)
    float *W1, *W2;           // updated when sgd
    float *dW1, *dW2;         // written when !sgd
    float *loss;              // nullable [1]
    float *step_loss;         // nullable
    int64_t step;
    float *epoch_loss;        // nullable
    int32_t epoch;
    int32_t first_in_epoch;
    Control *ctl;
};

size_t slot_stride_floats(int hidden);
int tile_rows_per_wg(int64_t nb);

hipError_t launch_forward(const Ctx &c, const float *X, int64_t n_rows, const int32_t *idx,
                          int64_t B, float *ypred);
hipError_t tile_step(const Ctx &c, const float *X, int64_t n_rows, const float *Y,
                     const int32_t *idx, int64_t idx_off, int64_t nb, const ReduceArgs &a);
hipError_t clear_control(const Ctx &c);
hipError_t clear_words(const Ctx &c, uint64_t *p, int64_t n);

// Host-loop strategies of the paper (hostloop.hip)
size_t hostloop_workspace_floats(int hidden, int64_t max_batch);
int hostloop_launches_per_step(int strategy);
hipError_t hostloop_step(const Ctx &c, const float *X, int64_t n_rows, const float *Y,
                         const int32_t *idx, int64_t idx_off, int64_t nb, const ReduceArgs &a);

// Persistent trainer
bool plan_train(int hidden, int64_t batch, TrainPlan *plan);
size_t persist_words_xch();
size_t persist_words_rs(int hidden);
size_t persist_words_ag(int hidden);
hipError_t launch_train(Ctx &c, TrainArgs &a);
hipError_t fill(const Ctx &c, float *p, int64_t n, float v);
void carve_workspace(Ctx &c, void *workspace, size_t need);

}  // namespace mlp

struct mlp_ctx : mlp::Ctx {};

// mlp_train_epochs on a context (api.hip), shared with the no-allocation entry point.
mlp_status train_epochs_ctx(mlp_ctx *c, const float *X, const float *Y, int64_t n, int64_t batch,
                            float lr, int32_t epochs, const int32_t *perm, int64_t max_steps,
                            float *epoch_loss, float *step_loss);
