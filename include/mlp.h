/*
 * mlp.h -- C ABI of the fused mini-batch SGD path for a d-h-1 ReLU/MSE
 * regression network with no biases, built for AMD Instinct MI355X (gfx950).
 *
 * The network and its training step are those of the paper's Sec. III:
 *   Z1 = X W1, H = ReLU(Z1), Ypred = H W2                (eqs. 11-13)
 *   L = (1/n_b) sum (Ypred - Y)^2                         (eq. 14)
 *   dZ2 = (2/n_b)(Ypred - Y), dW2 = H^T dZ2               (eqs. 15-16)
 *   dZ1 = (dZ2 W2^T) (.) [Z1 > 0], dW1 = X^T dZ1          (eqs. 17-18)
 *   W <- W - lr dW, both layers, after both gradients     (eq. 19)
 * with n_b the row count of the current mini-batch, mini-batch SGD over
 * epochs (Sec. II.A, Sec. III.A), and the last batch of an epoch keeping
 * its remainder rows.
 *
 * Conventions shared by every entry point
 *   - Every data pointer is a DEVICE pointer owned by the caller. The library
 *     never allocates or frees device memory; its scratch space is the
 *     caller's workspace buffer.
 *   - fp32 data, row-major. X is [n_rows x d_in]; Y is [n_rows]; W1 is
 *     [d_in x hidden] with rows = inputs (the paper's layout); W2 is
 *     [hidden] (the paper's hidden x 1 column, stored flat). Row indices and
 *     permutations are int32.
 *   - Calls are asynchronous on the context's stream. Argument errors are
 *     detected on the host before anything is enqueued; they return a
 *     negative status and leave weights and outputs untouched. Outputs are
 *     valid after the stream has been synchronised.
 *   - A row index outside [0, n_rows) is never dereferenced: the kernels read
 *     row 0 in its place and raise a sticky flag that mlp_check_errors()
 *     reports (results of that call are then meaningless).
 *   - Results are bitwise reproducible for identical inputs on one device:
 *     every reduction runs in a fixed order and no floating-point atomics are
 *     used.
 *   - One context per stream; a context is not re-entrant and calls on it
 *     must not overlap.
 */
#ifndef MLP_H_
#define MLP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mlp_ctx *mlp_t;

typedef enum {
    MLP_OK = 0,
    MLP_ERR_INVALID_ARG = -1,  /* null pointer, bad size, non-finite lr ...      */
    MLP_ERR_UNSUPPORTED = -2,  /* d_in != 32, d_out != 1, hidden not supported   */
    MLP_ERR_WORKSPACE = -3,    /* workspace too small or misaligned              */
    MLP_ERR_HIP = -4,          /* a HIP runtime call or kernel launch failed     */
    MLP_ERR_NONFINITE = -5,    /* a batch loss was NaN or infinite (diverged)    */
    MLP_ERR_INDEX = -6,        /* a kernel met a row index outside [0, n_rows)   */
    MLP_ERR_TIMEOUT = -7       /* a wait inside the training kernel timed out    */
} mlp_status;

/* Largest mini-batch any call accepts. */
#define MLP_MAX_BATCH (1 << 20)

/* Bytes of device workspace a context needs for the given shape. hidden must be
 * one of 32, 64, 128, 256, 512, 1024; d_in must be 32. Returns 0 for an
 * unsupported shape. The workspace must be 256-byte aligned. */
size_t mlp_workspace_bytes(int32_t d_in, int32_t hidden, int64_t max_batch);

/* Create a context bound to caller-owned weights and workspace.
 *   d_in      must be 32 (paper Sec. III.A input layer)
 *   hidden    32, 64, 128, 256 (the paper's net), 512 or 1024 (Sec. VI.C sweep)
 *   d_out     must be 1 (single regression output, Sec. III.A)
 *   max_batch largest batch later calls will use, 1..MLP_MAX_BATCH
 *   W1        [d_in x hidden] device fp32, updated in place by training calls
 *   W2        [hidden] device fp32, updated in place by training calls
 *   workspace device buffer of at least mlp_workspace_bytes(d_in, hidden,
 *             max_batch) bytes, 256-byte aligned, owned by the caller and kept
 *             alive for the life of the context
 *   stream    hipStream_t to enqueue on (NULL = the null stream)
 * Enqueues a clear of the whole workspace after the tile-path slots (control
 * words and exchange buffers) on `stream`; later calls must be ordered after
 * it (same stream, or a synchronisation). *out is set only on success. */
mlp_status mlp_init(mlp_t *out, int32_t d_in, int32_t hidden, int32_t d_out,
                    int64_t max_batch, float *W1, float *W2, void *workspace,
                    size_t ws_bytes, void *stream);

/* Rebind the stream later calls enqueue on. */
mlp_status mlp_set_stream(mlp_t ctx, void *stream);

/* Training strategies. They change how mlp_backward, mlp_sgd_step and
 * mlp_train_epochs compute (never what: every strategy computes eqs. 11-19 on
 * the same rows). MLP_STRATEGY_FUSED is the default; the others exist for the
 * strategy comparison of the paper's Sec. VI.B (Table I).
 *   FUSED     all steps of a call in one kernel launch (the persistent
 *             trainer); batch sizes it has no launch plan for run on TILE
 *   TILE      per step, one fused kernel (each workgroup a slice of the batch:
 *             forward, backward and its partial gradients in registers) and
 *             one fixed-order reduction that applies the update; host loop
 *   OPTIMIZED the paper's optimized strategy (Sec. V): LDS-tiled products on
 *             explicitly transposed operands, ReLU fused into the first
 *             product; one kernel per operation, intermediates in device
 *             memory, host loop
 *   BASELINE  the paper's baseline strategy (Sec. IV): one thread per output
 *             element reading global memory only, separate elementwise
 *             kernels, intermediates in device memory, host loop */
typedef enum {
    MLP_STRATEGY_FUSED = 0,
    MLP_STRATEGY_TILE = 1,
    MLP_STRATEGY_OPTIMIZED = 2,
    MLP_STRATEGY_BASELINE = 3
} mlp_strategy;

/* Bytes of device memory the strategy needs beyond the context's workspace,
 * for batches up to max_batch: 0 for FUSED and TILE; for OPTIMIZED and
 * BASELINE the intermediates of one step (about 4 * max_batch * (6 hidden +
 * 68) bytes). Returns 0 for an unsupported shape or strategy. */
size_t mlp_strategy_workspace_bytes(int32_t d_in, int32_t hidden, int64_t max_batch,
                                    int32_t strategy);

/* Select the strategy of later training calls on ctx. workspace (device,
 * 256-byte aligned, owned by the caller, kept alive while the strategy is
 * selected) must hold mlp_strategy_workspace_bytes(32, hidden, max_batch,
 * strategy) bytes for the context's max_batch; it may be NULL when that is 0.
 * On error the previous strategy stays selected. */
mlp_status mlp_set_strategy(mlp_t ctx, int32_t strategy, void *workspace, size_t ws_bytes);

/* Forward pass, eqs. (11)-(13): Ypred[t] = ReLU(X[r_t] W1) W2 for t < B, where
 * r_t = idx[t] (idx == NULL: r_t = t). X has n_rows rows. Ypred is [B].
 * B must be >= 1; it is not limited by max_batch. Weights are not changed. */
mlp_status mlp_forward(mlp_t ctx, const float *X, int64_t n_rows, const int32_t *idx,
                       int64_t B, float *Ypred);

/* Gradients of the batch loss at the current weights, eqs. (14)-(18), for the
 * B rows r_t (as in mlp_forward). Writes dW1 [d_in x hidden] and dW2 [hidden]
 * in the caller's layout (both include the 2/B factor of eq. 15) and, when
 * loss != NULL, loss[0] = batch MSE (eq. 14). 1 <= B <= max_batch. Weights are
 * not changed. */
mlp_status mlp_backward(mlp_t ctx, const float *X, int64_t n_rows, const float *Y,
                        const int32_t *idx, int64_t B, float *dW1, float *dW2,
                        float *loss);

/* One SGD step on the B rows r_t: the gradients of mlp_backward, then
 * W1 -= lr dW1 and W2 -= lr dW2 (eq. 19). loss (nullable) receives the batch
 * MSE before the update. 1 <= B <= max_batch; lr finite. */
mlp_status mlp_sgd_step(mlp_t ctx, const float *X, int64_t n_rows, const float *Y,
                        const int32_t *idx, int64_t B, float lr, float *loss);

/* Mini-batch SGD over epochs (Sec. II.A, Sec. III.A, eq. 19). Epoch e visits
 * rows perm[e*n + 0 .. n-1] in order (perm == NULL: rows 0..n-1 every epoch)
 * in ceil(n/batch) steps; the last step of an epoch takes the remainder rows
 * and scales by its own row count. X/Y have n rows.
 *   1 <= batch <= max_batch, epochs >= 1, lr finite
 *   max_steps   stop after this many steps in total (-1: run every epoch)
 *   epoch_loss  nullable [epochs]: sum of the epoch's squared residuals
 *               (each taken before its step's update) / n; entries of epochs
 *               cut short by max_steps hold the partial sum / n, later ones 0
 *   step_loss   nullable [steps run]: batch MSE of each step before its update
 * Each perm row must be a permutation of [0, n) (checked only for range). */
mlp_status mlp_train_epochs(mlp_t ctx, const float *X, const float *Y, int64_t n,
                            int64_t batch, float lr, int32_t epochs,
                            const int32_t *perm, int64_t max_steps,
                            float *epoch_loss, float *step_loss);

/* Synchronise the stream and report sticky kernel-side errors (MLP_ERR_INDEX,
 * MLP_ERR_TIMEOUT, MLP_ERR_NONFINITE) raised since the last check; clears them.
 * MLP_ERR_NONFINITE means some batch loss of a training or gradient call was
 * NaN or infinite (training diverged); the computation itself is not stopped,
 * and non-finite values propagate as fp32 arithmetic makes them. When several
 * errors were raised, the one reported is the last written. */
mlp_status mlp_check_errors(mlp_t ctx);

/* Timing of the training kernel. When enabled, mlp_train_epochs and
 * mlp_sgd_step bracket their training-kernel launches with HIP events on the
 * context's stream; mlp_last_kernel_ms synchronises on the end event and
 * returns the elapsed milliseconds of the most recent call's launches. */
mlp_status mlp_profile(mlp_t ctx, int32_t enable);
mlp_status mlp_last_kernel_ms(mlp_t ctx, float *ms);

/* Launch shape of an mlp_train_epochs call with these sizes under the selected
 * strategy: the number of workgroups of its main training kernel and the total
 * number of kernel launches the call enqueues (launch-count evidence for the
 * benchmark). */
mlp_status mlp_launch_info(mlp_t ctx, int64_t n, int64_t batch, int32_t epochs,
                           int32_t *workgroups, int64_t *launches);

/* Diagnostic: where the fused trainer's SGD step spends its cycles. With
 * MLP_TRACE=1 in the environment, a training call on the fused strategy makes
 * compute wave 0 and the first owner wave of every workgroup sum the core
 * cycles of each phase of the step (one SGD step, eqs. 11-19: forward operands,
 * forward, the exchange of partial outputs across groups, backward, the
 * reduction of the weight gradients, the update, the all-gather of the updated
 * weights; twelve phases) over the call's steps from the eighth on, into the
 * workspace. This call copies those sums of the context's last such call to
 * host memory: out[(wg * 2 + wave) * 16 + i], wave 0 = compute wave 0, 1 = the
 * owner wave; i = 0 steps summed, 1..12 the phases' cycles, 13 elapsed 100 MHz
 * ticks, 14 elapsed core cycles (their ratio is the clock), 15 unused.
 * out: host memory of max_words words (owned by the caller); *words receives
 * the number the last traced call wrote (0 if none). Copies min(max_words,
 * *words) words; blocks until the context's stream is idle. Errors:
 * MLP_ERR_INVALID_ARG for a null context or words pointer, MLP_ERR_HIP. */
mlp_status mlp_phase_cycles(mlp_t ctx, uint64_t *out, int64_t max_words, int64_t *words);

/* Release the host-side context (the caller still owns every device buffer). */
void mlp_destroy(mlp_t ctx);

/* mlp_train_epochs for callers that cannot allocate (code under stream capture,
 * tight serving loops, harnesses that forbid allocation): the same training
 * (the same kernels and launch sequence; results bitwise equal to
 * mlp_train_epochs on a context with the same weights and arguments), with no
 * context and no caller workspace. Its scratch is the library's own: a 16 MiB
 * device array per GPU, created with the library's code on that GPU and held
 * until the process ends. The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine, no host heap).
 *   hidden: 32, 64, 128 or 256 (larger nets need more than the 16 MiB scratch:
 *           MLP_ERR_WORKSPACE; other sizes MLP_ERR_UNSUPPORTED). d_in = 32, d_out = 1.
 *   W1 [32 x hidden], W2 [hidden]: device, caller-owned, updated in place.
 *   X, Y, n, batch (<= 2^20), lr, epochs, perm, max_steps, epoch_loss, step_loss:
 *           as mlp_train_epochs.
 *   status: nullable device int32; when given, receives the kernel-side sticky
 *           error of this call (0, MLP_ERR_INDEX, MLP_ERR_TIMEOUT or
 *           MLP_ERR_NONFINITE) once the call's work on the stream completes.
 *   stream: the HIP stream to enqueue on (NULL = the default stream).
 * Asynchronous: argument errors return synchronously before anything is
 * enqueued. Every call on a GPU shares that GPU's scratch, which keeps the last
 * call's contents: each call clears the control words it needs cleared, and
 * step tags continue across calls. Calls that overlap on one GPU (other streams
 * or threads without ordering) race on the scratch; calls on one stream do not. */
mlp_status mlp_train_epochs_static(int32_t hidden, float *W1, float *W2, const float *X,
                                   const float *Y, int64_t n, int64_t batch, float lr,
                                   int32_t epochs, const int32_t *perm, int64_t max_steps,
                                   float *epoch_loss, float *step_loss, int32_t *status,
                                   void *stream);

/* ---- Deeper networks: d_in-h-...-h-1 with L hidden layers ----------------------
 * The paper trains one hidden layer and names deeper networks as future work
 * (Sec. VII.B). These calls train the same kind of network with L hidden ReLU
 * layers of width h, by the chain rule of eqs. 11-19 applied layer by layer
 * (the layer index of eq. 9):
 *   H_0 = X, H_l = ReLU(H_{l-1} W_l) (l = 1..L), Ypred = H_L w_o,
 *   L = (1/n_b) sum (Ypred - Y)^2, dZ_o = (2/n_b)(Ypred - Y), dw_o = H_L^T dZ_o,
 *   dZ_l = dH_l (.) [Z_l > 0], dW_l = H_{l-1}^T dZ_l, dH_{l-1} = dZ_l W_l^T,
 *   every parameter -= lr * its gradient once all gradients are formed.
 * With L = 1 the network and its step are those of the calls above.
 * Parameters live in ONE flat fp32 device array owned by the caller:
 *   W_1 [d_in x h] row-major (rows = inputs), then W_2 ... W_L, each [h x h]
 *   row-major (rows = units of the layer below), then w_o [h].
 * Conventions (device pointers, asynchronous stream semantics, host-side
 * argument checks that leave parameters untouched, sticky index errors,
 * bitwise reproducibility, one context per stream) are those of the calls
 * above. Each SGD step is a sequence of kernel launches from the host (MFMA
 * GEMMs over the batch's activations in the workspace). */
typedef struct mlp_deep_ctx *mlp_deep_t;

/* Parameters of a d_in-h-...-h-1 net with `layers` hidden layers:
 * d_in h + (layers - 1) h^2 + h. 0 for an unsupported shape: d_in must be 32,
 * hidden a multiple of 64 in [64, 1024], layers in [1, 8]. */
int64_t mlp_deep_param_count(int32_t d_in, int32_t hidden, int32_t layers);

/* Workspace bytes for batches up to max_batch (the activations of every layer
 * for max_batch rows, gradient partials, control words); 0 if unsupported.
 * The workspace must be 256-byte aligned. */
size_t mlp_deep_workspace_bytes(int32_t d_in, int32_t hidden, int32_t layers, int64_t max_batch);

/* Create a context bound to caller-owned parameters (updated in place by
 * training calls) and workspace; d_out must be 1. Enqueues a clear of the
 * control words on `stream`. */
mlp_status mlp_deep_init(mlp_deep_t *out, int32_t d_in, int32_t hidden, int32_t layers,
                         int32_t d_out, int64_t max_batch, float *params, void *workspace,
                         size_t ws_bytes, void *stream);

/* Ypred[t] for rows r_t = idx[t] (idx == NULL: r_t = t), t < B; any B >= 1
 * (processed max_batch rows at a time). */
mlp_status mlp_deep_forward(mlp_deep_t ctx, const float *X, int64_t n_rows, const int32_t *idx,
                            int64_t B, float *Ypred);

/* Gradients of the batch loss at the current parameters into dparams (the
 * parameter layout, 2/B factor included); loss (nullable) = batch MSE.
 * 1 <= B <= max_batch. */
mlp_status mlp_deep_backward(mlp_deep_t ctx, const float *X, int64_t n_rows, const float *Y,
                             const int32_t *idx, int64_t B, float *dparams, float *loss);

/* One SGD step on the B rows r_t (the gradients of mlp_deep_backward, then
 * params -= lr * dparams); loss (nullable) = batch MSE before the update. */
mlp_status mlp_deep_sgd_step(mlp_deep_t ctx, const float *X, int64_t n_rows, const float *Y,
                             const int32_t *idx, int64_t B, float lr, float *loss);

/* Mini-batch SGD over epochs, with the schedule, permutations, tail batches and
 * loss outputs of mlp_train_epochs. */
mlp_status mlp_deep_train_epochs(mlp_deep_t ctx, const float *X, const float *Y, int64_t n,
                                 int64_t batch, float lr, int32_t epochs, const int32_t *perm,
                                 int64_t max_steps, float *epoch_loss, float *step_loss);

/* Synchronise and report (then clear) a sticky MLP_ERR_INDEX or MLP_ERR_NONFINITE
 * (as mlp_check_errors). */
mlp_status mlp_deep_check_errors(mlp_deep_t ctx);

/* HIP-event timing of the last mlp_deep_sgd_step / mlp_deep_train_epochs call
 * (all of its launches), as mlp_profile / mlp_last_kernel_ms. */
mlp_status mlp_deep_profile(mlp_deep_t ctx, int32_t enable);
mlp_status mlp_deep_last_kernel_ms(mlp_deep_t ctx, float *ms);

/* Release the host-side context. */
void mlp_deep_destroy(mlp_deep_t ctx);

/* Static description of a status code: any int32 value (a code that is not an
 * mlp_status gives "unknown status"). */
const char *mlp_status_string(int32_t status);

#ifdef __cplusplus
}
#endif
#endif /* MLP_H_ */
