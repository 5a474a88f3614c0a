// noalloc.hip -- mlp_train_epochs_static: mlp_train_epochs for callers that
// cannot allocate (code under stream capture, tight serving loops, harnesses
// that forbid allocation). Instead of a context and a caller-owned workspace it
// uses the library's own device scratch: a file-scope array, one copy per GPU,
// held until the process ends. The call allocates nothing (no hipMalloc, no
// hipFree, no allocating library routine, no host heap): it carves a context
// on the stack over the scratch and runs the same launch sequence, on the same
// kernels, as mlp_train_epochs.
//
// Every call on a GPU shares that GPU's scratch and finds it as the last call
// left it: each call clears the control words (sticky error, abort flag,
// registration counters) with a kernel on the caller's stream, and the step
// tags of the exchange words continue from the previous call on the device (the
// first call on a device clears every exchange word to tag 0). Calls that
// overlap on one GPU (different streams, or different threads without
// ordering) race on the scratch; calls on one stream are ordered.
#include <hip/hip_runtime.h>

#include <math.h>
#include <mutex>
#include <stdint.h>
#include <string.h>

#include "mlp.h"
#include "mlp_internal.h"

namespace mlp {

constexpr size_t STATIC_SCRATCH_BYTES = (size_t)16 << 20;   // 16 MiB per GPU
constexpr int STATIC_MAX_HIDDEN = 256;     // the largest net whose workspace fits
constexpr int STATIC_MAX_DEVICES = 64;

// The device scratch. In host code this name is a host-side stand-in, not a
// device address: its address on each device comes from hipGetSymbolAddress,
// called once per device with that device current, and only that address is
// passed to kernels and clears.
static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

struct StaticDevice {
    void *ptr = nullptr;      // the scratch's address on the device
    uint32_t tag_base = 1;    // first step tag of the next call
    int num_cu = 0;
};

static std::mutex g_mu;
static StaticDevice g_dev[STATIC_MAX_DEVICES];

// One layout of the scratch for every hidden size: the workspace of the largest
// net (control words, tile-path slots, then the exchange words), with this
// call's slot stride. The exchange words thus always sit at the same place,
// after every region that holds untagged data, and step tags rise across calls
// of any size: a word left by an earlier call never presents a current tag.
static void carve_static(mlp_ctx &c, void *ptr, int hidden) {
    c.hidden = STATIC_MAX_HIDDEN;
    carve_workspace(c, ptr, STATIC_SCRATCH_BYTES);   // exchange words to the scratch's end
    c.hidden = hidden;
    c.slot_stride = (int64_t)slot_stride_floats(hidden);
}

__global__ void k_copy_err(const Control *ctl, int32_t *status) {
    if (threadIdx.x == 0 && blockIdx.x == 0) status[0] = ctl->err;
}

}  // namespace mlp

using namespace mlp;

extern "C" mlp_status mlp_train_epochs_static(int32_t hidden, float *W1, float *W2,
                                              const float *X, const float *Y, int64_t n,
                                              int64_t batch, float lr, int32_t epochs,
                                              const int32_t *perm, int64_t max_steps,
                                              float *epoch_loss, float *step_loss,
                                              int32_t *status, void *stream) {
    if (!W1 || !W2 || !X || !Y || n < 1 || batch < 1 || batch > MLP_MAX_BATCH || epochs < 1 ||
        !isfinite(lr) || max_steps < -1 || (int64_t)epochs * n > ((int64_t)1 << 40))
        return MLP_ERR_INVALID_ARG;
    const size_t need = mlp_workspace_bytes(D_IN, hidden, batch);   // 0: unsupported hidden
    if (need == 0) return MLP_ERR_UNSUPPORTED;
    if (hidden > STATIC_MAX_HIDDEN ||
        mlp_workspace_bytes(D_IN, STATIC_MAX_HIDDEN, batch) > STATIC_SCRATCH_BYTES)
        return MLP_ERR_WORKSPACE;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return MLP_ERR_HIP;
    if (device < 0 || device >= STATIC_MAX_DEVICES) return MLP_ERR_UNSUPPORTED;

    std::lock_guard<std::mutex> lock(g_mu);
    StaticDevice &d = g_dev[device];
    mlp_ctx c;                          // on the stack: nothing is allocated
    c.hidden = hidden;
    c.max_batch = batch;
    c.W1 = W1;
    c.W2 = W2;
    c.stream = (hipStream_t)stream;
    c.device = device;
    const bool first = d.ptr == nullptr;
    if (first) {
        // set-up on this device, with it current: the scratch's device address
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return MLP_ERR_HIP;
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) !=
            hipSuccess)
            return MLP_ERR_HIP;
        d.num_cu = cus;
        d.tag_base = 1;
        carve_static(c, ptr, hidden);
        // every exchange word to tag 0 before the first call's tags start at 1
        if (clear_words(c, c.xch, c.xch_words) != hipSuccess) return MLP_ERR_HIP;
        d.ptr = ptr;
    } else {
        carve_static(c, d.ptr, hidden);
    }
    c.num_cu = d.num_cu;
    c.tag_base = d.tag_base;   // a range that would wrap clears every exchange word
    if (clear_control(c) != hipSuccess) return MLP_ERR_HIP;
    const mlp_status st = train_epochs_ctx(&c, X, Y, n, batch, lr, epochs, perm, max_steps,
                                           epoch_loss, step_loss);
    d.tag_base = c.tag_base;
    if (st != MLP_OK) return st;
    if (status) {
        hipLaunchKernelGGL(k_copy_err, dim3(1), dim3(64), 0, c.stream, c.ctl, status);
        if (hipGetLastError() != hipSuccess) return MLP_ERR_HIP;
    }
    return MLP_OK;
}
