// api.hip -- host side of the C ABI declared in include/mlp.h: argument
// validation, workspace carving, and the launch sequence of each call.
#include <hip/hip_runtime.h>

#include <math.h>
#include <new>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "mlp.h"
#include "mlp_internal.h"

using namespace mlp;

namespace mlp {

size_t slot_stride_floats(int hidden) {
    // [dW1 (32 h) | dW2 (h) | sse (1)], padded to 64 floats (256 B).
    size_t n = (size_t)(D_IN + 1) * hidden + 1;
    return (n + 63) / 64 * 64;
}

}  // namespace mlp

static bool hidden_supported(int32_t h) {
    return h == 32 || h == 64 || h == 128 || h == 256 || h == 512 || h == 1024;
}

static size_t round256(size_t b) { return (b + 255) / 256 * 256; }

extern "C" size_t mlp_workspace_bytes(int32_t d_in, int32_t hidden, int64_t max_batch) {
    if (d_in != D_IN || !hidden_supported(hidden) || max_batch < 1 || max_batch > MLP_MAX_BATCH)
        return 0;
    size_t b = CTL_BYTES;
    b += round256(sizeof(float) * slot_stride_floats(hidden) * TILE_SLOTS);
    b += round256(sizeof(uint64_t) * persist_words_xch());
    b += round256(sizeof(uint64_t) * persist_words_rs(hidden));
    b += round256(sizeof(uint64_t) * persist_words_ag(hidden));
    return b;
}

extern "C" const char *mlp_status_string(int32_t s) {
    switch (s) {
    case MLP_OK: return "ok";
    case MLP_ERR_INVALID_ARG: return "invalid argument";
    case MLP_ERR_UNSUPPORTED: return "unsupported shape";
    case MLP_ERR_WORKSPACE: return "workspace too small or misaligned";
    case MLP_ERR_HIP: return "HIP runtime error";
    case MLP_ERR_INDEX: return "row index out of range";
    case MLP_ERR_TIMEOUT: return "a wait in the training kernel timed out";
    case MLP_ERR_NONFINITE: return "a batch loss was NaN or infinite";
    }
    return "unknown status";
}

static mlp_status hip_status(hipError_t e) { return e == hipSuccess ? MLP_OK : MLP_ERR_HIP; }

namespace mlp {

// Pointers of a context into a workspace of `need` bytes (mlp_workspace_bytes):
// control words, tile-path slots, then the trainer's three exchange buffers.
void carve_workspace(Ctx &c, void *workspace, size_t need) {
    char *ws = (char *)workspace;
    c.ctl = (Control *)ws;
    ws += CTL_BYTES;
    c.slot_stride = (int64_t)slot_stride_floats(c.hidden);
    c.slots = (float *)ws;
    ws += round256(sizeof(float) * c.slot_stride * TILE_SLOTS);
    c.xch = (uint64_t *)ws;
    ws += round256(sizeof(uint64_t) * persist_words_xch());
    c.rs = (uint64_t *)ws;
    ws += round256(sizeof(uint64_t) * persist_words_rs(c.hidden));
    c.ag = (uint64_t *)ws;
    c.xch_words = (int64_t)(((char *)workspace + need) - (char *)c.xch) / 8;
}

}  // namespace mlp

extern "C" mlp_status mlp_init(mlp_t *out, int32_t d_in, int32_t hidden, int32_t d_out,
                               int64_t max_batch, float *W1, float *W2, void *workspace,
                               size_t ws_bytes, void *stream) {
    if (!out || !W1 || !W2 || !workspace) return MLP_ERR_INVALID_ARG;
    if (d_in != D_IN || d_out != 1 || !hidden_supported(hidden)) return MLP_ERR_UNSUPPORTED;
    if (max_batch < 1 || max_batch > MLP_MAX_BATCH) return MLP_ERR_INVALID_ARG;
    const size_t need = mlp_workspace_bytes(d_in, hidden, max_batch);
    if (ws_bytes < need || ((uintptr_t)workspace & 255u)) return MLP_ERR_WORKSPACE;
    mlp_ctx *c = new (std::nothrow) mlp_ctx();
    if (!c) return MLP_ERR_HIP;
    c->hidden = hidden;
    c->max_batch = max_batch;
    c->W1 = W1;
    c->W2 = W2;
    carve_workspace(*c, workspace, need);
    c->stream = (hipStream_t)stream;
    // Exchange words carry (value, step tag); tags of this context start at 1, so
    // every word is cleared to tag 0 first: memory reused from an earlier
    // context can never present a current tag.
    const int64_t words = c->xch_words;
    // test hook: the first step tag of this context (exercises the tag wrap)
    if (const char *tb = getenv("MLP_TAG_BASE")) c->tag_base = (uint32_t)strtoul(tb, nullptr, 10);
    if (hipGetDevice(&c->device) != hipSuccess ||
        hipDeviceGetAttribute(&c->num_cu, hipDeviceAttributeMultiprocessorCount, c->device) !=
            hipSuccess ||
        clear_control(*c) != hipSuccess || clear_words(*c, c->xch, words) != hipSuccess) {
        delete c;
        return MLP_ERR_HIP;
    }
    *out = c;
    return MLP_OK;
}

static bool strategy_valid(int32_t s) {
    return s == MLP_STRATEGY_FUSED || s == MLP_STRATEGY_TILE || s == MLP_STRATEGY_OPTIMIZED ||
           s == MLP_STRATEGY_BASELINE;
}

static bool strategy_hostloop(int32_t s) {
    return s == MLP_STRATEGY_OPTIMIZED || s == MLP_STRATEGY_BASELINE;
}

extern "C" size_t mlp_strategy_workspace_bytes(int32_t d_in, int32_t hidden, int64_t max_batch,
                                               int32_t strategy) {
    if (d_in != D_IN || !hidden_supported(hidden) || max_batch < 1 || max_batch > MLP_MAX_BATCH ||
        !strategy_hostloop(strategy))
        return 0;
    return round256(sizeof(float) * hostloop_workspace_floats(hidden, max_batch));
}

extern "C" mlp_status mlp_set_strategy(mlp_t c, int32_t strategy, void *workspace,
                                       size_t ws_bytes) {
    if (!c || !strategy_valid(strategy)) return MLP_ERR_INVALID_ARG;
    if (strategy_hostloop(strategy)) {
        const size_t need = mlp_strategy_workspace_bytes(D_IN, c->hidden, c->max_batch, strategy);
        if (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255u)) return MLP_ERR_WORKSPACE;
        c->hl_ws = (float *)workspace;
        c->hl_max_batch = c->max_batch;
    } else {
        c->hl_ws = nullptr;
        c->hl_max_batch = 0;
    }
    c->strategy = strategy;
    return MLP_OK;
}

extern "C" mlp_status mlp_set_stream(mlp_t c, void *stream) {
    if (!c) return MLP_ERR_INVALID_ARG;
    c->stream = (hipStream_t)stream;
    return MLP_OK;
}

extern "C" void mlp_destroy(mlp_t c) {
    if (!c) return;
    if (c->ev0) (void)hipEventDestroy(c->ev0);
    if (c->ev1) (void)hipEventDestroy(c->ev1);
    delete c;
}

extern "C" mlp_status mlp_forward(mlp_t c, const float *X, int64_t n_rows, const int32_t *idx,
                                  int64_t B, float *Ypred) {
    if (!c || !X || !Ypred || B < 1 || n_rows < 1) return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    return hip_status(launch_forward(*c, X, n_rows, idx, B, Ypred));
}

static ReduceArgs base_args(const mlp_ctx *c, int64_t nb) {
    ReduceArgs a;
    memset(&a, 0, sizeof(a));
    a.inv_nb = (float)(1.0 / (double)nb);
    a.W1 = c->W1;
    a.W2 = c->W2;
    a.ctl = c->ctl;
    return a;
}

static void prof_begin(mlp_ctx *c) {
    if (!c->profile) return;
    if (!c->ev0) (void)hipEventCreate(&c->ev0);
    if (!c->ev1) (void)hipEventCreate(&c->ev1);
    (void)hipEventRecord(c->ev0, c->stream);
}

static void prof_end(mlp_ctx *c) {
    if (!c->profile) return;
    (void)hipEventRecord(c->ev1, c->stream);
    c->ev_valid = true;
}

// Under the FUSED strategy the persistent trainer runs every SGD step of a call
// in one launch; the tile path (two launches per step) serves batches the
// trainer's plan cannot hold, and every call under the TILE strategy.
static bool use_persistent(const mlp_ctx *c, int64_t batch, TrainPlan *pl) {
    if (c->strategy != MLP_STRATEGY_FUSED) return false;
    return plan_train(c->hidden, batch, pl);
}

// One host-driven step under the TILE, OPTIMIZED or BASELINE strategy.
static hipError_t host_step(const mlp_ctx *c, const float *X, int64_t n_rows, const float *Y,
                            const int32_t *idx, int64_t idx_off, int64_t nb, const ReduceArgs &a) {
    if (strategy_hostloop(c->strategy)) return hostloop_step(*c, X, n_rows, Y, idx, idx_off, nb, a);
    return tile_step(*c, X, n_rows, Y, idx, idx_off, nb, a);
}

static TrainArgs train_args(const mlp_ctx *c, const TrainPlan &pl) {
    TrainArgs a;
    memset(&a, 0, sizeof(a));
    a.hidden = c->hidden;
    a.W1 = c->W1;
    a.W2 = c->W2;
    a.plan = pl;
    return a;
}

extern "C" mlp_status mlp_backward(mlp_t c, const float *X, int64_t n_rows, const float *Y,
                                   const int32_t *idx, int64_t B, float *dW1, float *dW2,
                                   float *loss) {
    if (!c || !X || !Y || !dW1 || !dW2 || B < 1 || B > c->max_batch || n_rows < 1)
        return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    TrainPlan pl;
    if (use_persistent(c, B, &pl)) {
        TrainArgs t = train_args(c, pl);
        t.X = X; t.Y = Y; t.n_rows = n_rows; t.perm = idx;
        t.n = B; t.batch = B; t.steps = 1; t.epochs = 1;
        t.inv_n = (float)(1.0 / (double)B);
        t.mode = 1;
        t.dW1 = dW1; t.dW2 = dW2; t.loss = loss;
        return hip_status(launch_train(*c, t));
    }
    ReduceArgs a = base_args(c, B);
    a.sgd = 0;
    a.dW1 = dW1;
    a.dW2 = dW2;
    a.loss = loss;
    return hip_status(host_step(c, X, n_rows, Y, idx, 0, B, a));
}

extern "C" mlp_status mlp_sgd_step(mlp_t c, const float *X, int64_t n_rows, const float *Y,
                                   const int32_t *idx, int64_t B, float lr, float *loss) {
    if (!c || !X || !Y || B < 1 || B > c->max_batch || n_rows < 1 || !isfinite(lr))
        return MLP_ERR_INVALID_ARG;
    if (!idx && B > n_rows) return MLP_ERR_INVALID_ARG;
    TrainPlan pl;
    prof_begin(c);
    mlp_status st;
    if (use_persistent(c, B, &pl)) {
        TrainArgs t = train_args(c, pl);
        t.X = X; t.Y = Y; t.n_rows = n_rows; t.perm = idx;
        t.n = B; t.batch = B; t.steps = 1; t.epochs = 1;
        t.inv_n = (float)(1.0 / (double)B);
        t.lr = lr; t.mode = 0; t.loss = loss;
        st = hip_status(launch_train(*c, t));
    } else {
        ReduceArgs a = base_args(c, B);
        a.sgd = 1;
        a.lr = lr;
        a.loss = loss;
        st = hip_status(host_step(c, X, n_rows, Y, idx, 0, B, a));
    }
    prof_end(c);
    return st;
}

extern "C" mlp_status mlp_train_epochs(mlp_t c, const float *X, const float *Y, int64_t n,
                                       int64_t batch, float lr, int32_t epochs,
                                       const int32_t *perm, int64_t max_steps,
                                       float *epoch_loss, float *step_loss) {
    return train_epochs_ctx(c, X, Y, n, batch, lr, epochs, perm, max_steps, epoch_loss, step_loss);
}

mlp_status train_epochs_ctx(mlp_ctx *c, const float *X, const float *Y, int64_t n, int64_t batch,
                            float lr, int32_t epochs, const int32_t *perm, int64_t max_steps,
                            float *epoch_loss, float *step_loss) {
    if (!c || !X || !Y || n < 1 || batch < 1 || batch > c->max_batch || epochs < 1 ||
        !isfinite(lr) || max_steps < -1)
        return MLP_ERR_INVALID_ARG;
    if ((int64_t)epochs * n > ((int64_t)1 << 40)) return MLP_ERR_INVALID_ARG;
    const int64_t spe_all = (n + batch - 1) / batch;
    int64_t total = spe_all * (int64_t)epochs;
    if (max_steps >= 0 && max_steps < total) total = max_steps;
    TrainPlan pl;
    if (total > 0 && total < ((int64_t)1 << 30) && use_persistent(c, batch, &pl)) {
        TrainArgs t = train_args(c, pl);
        t.X = X; t.Y = Y; t.n_rows = n; t.perm = perm;
        t.n = n; t.batch = batch; t.steps = total; t.epochs = epochs;
        t.inv_n = (float)(1.0 / (double)n);
        t.lr = lr; t.mode = 0;
        t.step_loss = step_loss; t.epoch_loss = epoch_loss;
        prof_begin(c);
        mlp_status st = hip_status(launch_train(*c, t));
        prof_end(c);
        return st;
    }
    hipError_t e = hipSuccess;
    if (epoch_loss) e = fill(*c, epoch_loss, epochs, 0.0f);
    if (e != hipSuccess) return MLP_ERR_HIP;
    const int64_t spe = (n + batch - 1) / batch;
    int64_t step = 0;
    prof_begin(c);
    for (int32_t ep = 0; ep < epochs && e == hipSuccess; ++ep) {
        for (int64_t s = 0; s < spe; ++s) {
            if (max_steps >= 0 && step >= max_steps) break;
            const int64_t off = s * batch;
            const int64_t nb = n - off < batch ? n - off : batch;
            ReduceArgs a = base_args(c, nb);
            a.sgd = 1;
            a.lr = lr;
            a.inv_n = (float)(1.0 / (double)n);
            a.step_loss = step_loss;
            a.step = step;
            a.epoch_loss = epoch_loss;
            a.epoch = ep;
            a.first_in_epoch = s == 0;
            const int32_t *ix = perm ? perm + (int64_t)ep * n : nullptr;
            e = host_step(c, X, n, Y, ix, off, nb, a);
            if (e != hipSuccess) break;
            ++step;
        }
    }
    prof_end(c);
    return hip_status(e);
}

extern "C" mlp_status mlp_check_errors(mlp_t c) {
    if (!c) return MLP_ERR_INVALID_ARG;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return MLP_ERR_HIP;
    int32_t err = 0;
    if (hipMemcpy(&err, &c->ctl->err, sizeof(err), hipMemcpyDeviceToHost) != hipSuccess)
        return MLP_ERR_HIP;
    if (err) {
        if (clear_control(*c) != hipSuccess || hipStreamSynchronize(c->stream) != hipSuccess)
            return MLP_ERR_HIP;
        if (err == MLP_ERR_TIMEOUT || err == MLP_ERR_NONFINITE) return (mlp_status)err;
        return MLP_ERR_INDEX;
    }
    return MLP_OK;
}

extern "C" mlp_status mlp_profile(mlp_t c, int32_t enable) {
    if (!c) return MLP_ERR_INVALID_ARG;
    c->profile = enable != 0;
    c->ev_valid = false;
    return MLP_OK;
}

extern "C" mlp_status mlp_last_kernel_ms(mlp_t c, float *ms) {
    if (!c || !ms) return MLP_ERR_INVALID_ARG;
    if (!c->ev_valid) return MLP_ERR_INVALID_ARG;
    if (hipEventSynchronize(c->ev1) != hipSuccess) return MLP_ERR_HIP;
    return hip_status(hipEventElapsedTime(ms, c->ev0, c->ev1));
}

extern "C" mlp_status mlp_phase_cycles(mlp_t c, uint64_t *out, int64_t max_words,
                                       int64_t *words) {
    if (!c || !words || max_words < 0) return MLP_ERR_INVALID_ARG;
    *words = c->phase_words;
    const int64_t n = c->phase_words < max_words ? c->phase_words : max_words;
    if (n <= 0 || !out) return MLP_OK;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return MLP_ERR_HIP;
    return hip_status(hipMemcpy(out, c->slots, sizeof(uint64_t) * (size_t)n, hipMemcpyDeviceToHost));
}

extern "C" mlp_status mlp_launch_info(mlp_t c, int64_t n, int64_t batch, int32_t epochs,
                                      int32_t *workgroups, int64_t *launches) {
    if (!c || !workgroups || !launches || n < 1 || batch < 1 || epochs < 1)
        return MLP_ERR_INVALID_ARG;
    TrainPlan pl;
    if (use_persistent(c, batch, &pl)) {
        *workgroups = pl.grid;
        *launches = 1;
        return MLP_OK;
    }
    const int64_t steps = ((n + batch - 1) / batch) * (int64_t)epochs;
    if (strategy_hostloop(c->strategy)) {
        // the largest product grid: 16 x 16 blocks over [batch x hidden]
        *workgroups = (int32_t)(((batch + 15) / 16) * ((c->hidden + 15) / 16));
        *launches = hostloop_launches_per_step(c->strategy) * steps + 1;
        return MLP_OK;
    }
    const int R = tile_rows_per_wg(batch);
    *workgroups = (int32_t)((batch + R - 1) / R);
    *launches = 2 * steps + 1;
    return MLP_OK;
}
