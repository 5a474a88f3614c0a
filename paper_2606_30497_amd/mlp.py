"""Thin ctypes binding of libmlp.so (include/mlp.h).

Argument marshalling only: every step of the training path runs in the HIP
kernels of libmlp.so. torch supplies device memory and the stream; tensors are
checked for device, dtype, shape and contiguity, then their data pointers are
passed through. There is no CPU fallback: if the library or a GPU is missing,
every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

from . import build as _build

D_IN = 32
HIDDEN_SIZES = (32, 64, 128, 256, 512, 1024)
MAX_BATCH = 1 << 20

MLP_OK = 0
STATUS = {0: "MLP_OK", -1: "MLP_ERR_INVALID_ARG", -2: "MLP_ERR_UNSUPPORTED",
          -3: "MLP_ERR_WORKSPACE", -4: "MLP_ERR_HIP", -5: "MLP_ERR_NONFINITE",
          -6: "MLP_ERR_INDEX", -7: "MLP_ERR_TIMEOUT"}

STRATEGY_FUSED, STRATEGY_TILE, STRATEGY_OPTIMIZED, STRATEGY_BASELINE = 0, 1, 2, 3
STRATEGIES = {"fused": STRATEGY_FUSED, "tile": STRATEGY_TILE, "optimized": STRATEGY_OPTIMIZED,
              "baseline": STRATEGY_BASELINE}

EXPORTS = ("mlp_workspace_bytes", "mlp_init", "mlp_set_stream", "mlp_strategy_workspace_bytes",
           "mlp_set_strategy", "mlp_forward", "mlp_backward",
           "mlp_sgd_step", "mlp_train_epochs", "mlp_check_errors", "mlp_profile",
           "mlp_last_kernel_ms", "mlp_launch_info", "mlp_phase_cycles", "mlp_destroy",
           "mlp_train_epochs_static", "mlp_status_string",
           "mlp_deep_param_count", "mlp_deep_workspace_bytes", "mlp_deep_init", "mlp_deep_forward",
           "mlp_deep_backward", "mlp_deep_sgd_step", "mlp_deep_train_epochs",
           "mlp_deep_check_errors", "mlp_deep_profile", "mlp_deep_last_kernel_ms",
           "mlp_deep_destroy")


class MLPError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (fn, STATUS.get(status, "?"), status))


_lib = None

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float


def library_path() -> str:
    """The in-tree libmlp.so, or another build of it that MLP_LIBRARY names."""
    return os.environ.get("MLP_LIBRARY") or _build.LIB


def load(require_built: bool = True):
    """Load libmlp.so (after torch, so that both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        if require_built or path != _build.LIB:
            raise RuntimeError("%s is not built (run __graft_entry__.build())" % path)
        _build.build()
    lib = ctypes.CDLL(path)
    sig = {
        "mlp_workspace_bytes": (ctypes.c_size_t, [_i32, _i32, _i64]),
        "mlp_init": (ctypes.c_int, [ctypes.POINTER(_vp), _i32, _i32, _i32, _i64, _vp, _vp, _vp,
                                    ctypes.c_size_t, _vp]),
        "mlp_set_stream": (ctypes.c_int, [_vp, _vp]),
        "mlp_strategy_workspace_bytes": (ctypes.c_size_t, [_i32, _i32, _i64, _i32]),
        "mlp_set_strategy": (ctypes.c_int, [_vp, _i32, _vp, ctypes.c_size_t]),
        "mlp_forward": (ctypes.c_int, [_vp, _vp, _i64, _vp, _i64, _vp]),
        "mlp_backward": (ctypes.c_int, [_vp, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp]),
        "mlp_sgd_step": (ctypes.c_int, [_vp, _vp, _i64, _vp, _vp, _i64, _f32, _vp]),
        "mlp_train_epochs": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i64, _f32, _i32, _vp, _i64,
                                            _vp, _vp]),
        "mlp_check_errors": (ctypes.c_int, [_vp]),
        "mlp_profile": (ctypes.c_int, [_vp, _i32]),
        "mlp_last_kernel_ms": (ctypes.c_int, [_vp, ctypes.POINTER(_f32)]),
        "mlp_launch_info": (ctypes.c_int, [_vp, _i64, _i64, _i32, ctypes.POINTER(_i32),
                                           ctypes.POINTER(_i64)]),
        "mlp_phase_cycles": (ctypes.c_int, [_vp, _vp, _i64, ctypes.POINTER(_i64)]),
        "mlp_train_epochs_static": (ctypes.c_int, [_i32, _vp, _vp, _vp, _vp, _i64, _i64, _f32, _i32,
                                                   _vp, _i64, _vp, _vp, _vp, _vp]),
        "mlp_destroy": (None, [_vp]),
        "mlp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "mlp_deep_param_count": (_i64, [_i32, _i32, _i32]),
        "mlp_deep_workspace_bytes": (ctypes.c_size_t, [_i32, _i32, _i32, _i64]),
        "mlp_deep_init": (ctypes.c_int, [ctypes.POINTER(_vp), _i32, _i32, _i32, _i32, _i64, _vp,
                                         _vp, ctypes.c_size_t, _vp]),
        "mlp_deep_forward": (ctypes.c_int, [_vp, _vp, _i64, _vp, _i64, _vp]),
        "mlp_deep_backward": (ctypes.c_int, [_vp, _vp, _i64, _vp, _vp, _i64, _vp, _vp]),
        "mlp_deep_sgd_step": (ctypes.c_int, [_vp, _vp, _i64, _vp, _vp, _i64, _f32, _vp]),
        "mlp_deep_train_epochs": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i64, _f32, _i32, _vp, _i64,
                                                 _vp, _vp]),
        "mlp_deep_check_errors": (ctypes.c_int, [_vp]),
        "mlp_deep_profile": (ctypes.c_int, [_vp, _i32]),
        "mlp_deep_last_kernel_ms": (ctypes.c_int, [_vp, ctypes.POINTER(_f32)]),
        "mlp_deep_destroy": (None, [_vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(fn, status):
    if status != MLP_OK:
        raise MLPError(fn, status)


def _dev(t, name, dtype=torch.float32, numel=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s" % (name, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if numel is not None and t.numel() < numel:
        raise ValueError("%s has %d elements, needs %d" % (name, t.numel(), numel))
    return t.data_ptr()


def mlp_workspace_bytes(d_in: int, hidden: int, max_batch: int) -> int:
    return int(load().mlp_workspace_bytes(d_in, hidden, max_batch))


class Context:
    """A library context bound to caller-owned W1, W2 and workspace tensors."""

    def __init__(self, handle, W1, W2, workspace, max_batch):
        self.handle = handle
        self.W1, self.W2, self.workspace = W1, W2, workspace
        self.max_batch = max_batch
        self.hidden = W1.shape[1]
        self.strategy_workspace = None

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and _lib is not None:
            _lib.mlp_destroy(h)


def mlp_init(W1: torch.Tensor, W2: torch.Tensor, max_batch: int, workspace=None,
             stream=None) -> Context:
    """Create a context. W1 [32, h] and W2 [h] (or [h, 1]) are updated in place."""
    lib = load()
    if W1.dim() != 2:
        raise ValueError("W1 must be [d_in, hidden]")
    d_in, h = W1.shape
    _dev(W1, "W1")
    _dev(W2, "W2", numel=h)
    need = lib.mlp_workspace_bytes(d_in, h, max_batch)
    if need == 0:
        raise MLPError("mlp_workspace_bytes", -2)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=W1.device)
    _dev(workspace, "workspace", dtype=torch.uint8, numel=need)
    if stream is None:
        stream = torch.cuda.current_stream(W1.device).cuda_stream
    handle = _vp()
    _check("mlp_init", lib.mlp_init(ctypes.byref(handle), d_in, h, 1, max_batch, W1.data_ptr(),
                                    W2.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                    stream))
    return Context(handle, W1, W2, workspace, max_batch)


def mlp_set_stream(ctx: Context, stream) -> None:
    _check("mlp_set_stream", load().mlp_set_stream(ctx.handle, stream))


def mlp_strategy_workspace_bytes(d_in: int, hidden: int, max_batch: int, strategy: int) -> int:
    return int(load().mlp_strategy_workspace_bytes(d_in, hidden, max_batch, strategy))


def mlp_set_strategy(ctx: Context, strategy, workspace=None) -> None:
    """Select the training strategy (a name of STRATEGIES or its code); allocates
    the strategy workspace as a torch tensor when none is given."""
    code = STRATEGIES[strategy] if isinstance(strategy, str) else int(strategy)
    need = mlp_strategy_workspace_bytes(D_IN, ctx.hidden, ctx.max_batch, code)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=ctx.W1.device)
    ptr = _dev(workspace, "workspace", dtype=torch.uint8, numel=need) if workspace is not None else None
    nbytes = workspace.numel() if workspace is not None else 0
    _check("mlp_set_strategy", load().mlp_set_strategy(ctx.handle, code, ptr, nbytes))
    ctx.strategy_workspace = workspace


def _rows(idx, B, name="idx"):
    if idx is None:
        return None
    return _dev(idx, name, dtype=torch.int32, numel=B)


def mlp_forward(ctx: Context, X, idx=None, B=None, out=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    if out is None:
        out = torch.empty(B, dtype=torch.float32, device=X.device)
    _check("mlp_forward", load().mlp_forward(ctx.handle, X.data_ptr(), n_rows, _rows(idx, B), B,
                                             _dev(out, "Ypred", numel=B)))
    return out


def mlp_backward(ctx: Context, X, Y, idx=None, B=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    _dev(Y, "Y", numel=n_rows)
    dW1 = torch.empty_like(ctx.W1)
    dW2 = torch.empty(ctx.hidden, dtype=torch.float32, device=X.device)
    loss = torch.empty(1, dtype=torch.float32, device=X.device)
    _check("mlp_backward", load().mlp_backward(ctx.handle, X.data_ptr(), n_rows, Y.data_ptr(),
                                               _rows(idx, B), B, dW1.data_ptr(), dW2.data_ptr(),
                                               loss.data_ptr()))
    return dW1, dW2, loss


def mlp_sgd_step(ctx: Context, X, Y, lr, idx=None, B=None, loss=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    _dev(Y, "Y", numel=n_rows)
    lp = _dev(loss, "loss", numel=1) if loss is not None else None
    _check("mlp_sgd_step", load().mlp_sgd_step(ctx.handle, X.data_ptr(), n_rows, Y.data_ptr(),
                                               _rows(idx, B), B, float(lr), lp))
    return loss


def mlp_train_epochs(ctx: Context, X, Y, batch, lr, epochs, perm=None, max_steps=-1,
                     epoch_loss=None, step_loss=None):
    n = X.shape[0]
    _dev(X, "X", numel=n * D_IN)
    _dev(Y, "Y", numel=n)
    pp = _dev(perm, "perm", dtype=torch.int32, numel=epochs * n) if perm is not None else None
    ep = _dev(epoch_loss, "epoch_loss", numel=epochs) if epoch_loss is not None else None
    steps = -(-n // batch) * epochs
    if max_steps >= 0:
        steps = min(steps, max_steps)
    sp = _dev(step_loss, "step_loss", numel=steps) if step_loss is not None else None
    _check("mlp_train_epochs", load().mlp_train_epochs(ctx.handle, X.data_ptr(), Y.data_ptr(), n,
                                                       batch, float(lr), epochs, pp, max_steps,
                                                       ep, sp))


def mlp_train_epochs_static(W1, W2, X, Y, batch, lr, epochs, perm=None, max_steps=-1,
                            epoch_loss=None, step_loss=None, status=None, stream=None):
    """mlp_train_epochs without a context: the library's own per-GPU scratch, no
    allocation in the call. W1 [32, h], W2 [h] are updated in place; status
    (nullable int32 [1]) receives the call's kernel-side error word."""
    if W1.dim() != 2:
        raise ValueError("W1 must be [d_in, hidden]")
    h = W1.shape[1]
    n = X.shape[0]
    _dev(W1, "W1")
    _dev(W2, "W2", numel=h)
    _dev(X, "X", numel=n * D_IN)
    _dev(Y, "Y", numel=n)
    pp = _dev(perm, "perm", dtype=torch.int32, numel=epochs * n) if perm is not None else None
    ep = _dev(epoch_loss, "epoch_loss", numel=epochs) if epoch_loss is not None else None
    steps = -(-n // batch) * epochs
    if max_steps >= 0:
        steps = min(steps, max_steps)
    sp = _dev(step_loss, "step_loss", numel=steps) if step_loss is not None else None
    stp = _dev(status, "status", dtype=torch.int32, numel=1) if status is not None else None
    if stream is None:
        stream = torch.cuda.current_stream(W1.device).cuda_stream
    _check("mlp_train_epochs_static",
           load().mlp_train_epochs_static(h, W1.data_ptr(), W2.data_ptr(), X.data_ptr(),
                                          Y.data_ptr(), n, batch, float(lr), epochs, pp,
                                          max_steps, ep, sp, stp, stream))


def mlp_check_errors(ctx: Context) -> None:
    _check("mlp_check_errors", load().mlp_check_errors(ctx.handle))


def mlp_profile(ctx: Context, enable: bool) -> None:
    _check("mlp_profile", load().mlp_profile(ctx.handle, 1 if enable else 0))


def mlp_last_kernel_ms(ctx: Context) -> float:
    ms = _f32(0.0)
    _check("mlp_last_kernel_ms", load().mlp_last_kernel_ms(ctx.handle, ctypes.byref(ms)))
    return float(ms.value)


def mlp_launch_info(ctx: Context, n, batch, epochs):
    wg = _i32(0)
    launches = _i64(0)
    _check("mlp_launch_info", load().mlp_launch_info(ctx.handle, n, batch, epochs,
                                                     ctypes.byref(wg), ctypes.byref(launches)))
    return int(wg.value), int(launches.value)


PHASE_NAMES = ("forward operands", "forward", "exchange A wait, tile 0",
               "residual tile 0 + exchange A wait, tile 1", "residual + backward + P to LDS",
               "P barrier", "exchange B stores", "exchange B wait", "update + exchange C stores",
               "owners barrier", "exchange C gather", "step barrier")


def mlp_phase_cycles(ctx: Context):
    """Phase-cycle sums of the context's last fused-trainer call made with
    MLP_TRACE=1 (see include/mlp.h): an int64 array [workgroups, 2, 16], or None
    when no traced call wrote any."""
    import numpy as np
    words = _i64(0)
    _check("mlp_phase_cycles", load().mlp_phase_cycles(ctx.handle, None, 0, ctypes.byref(words)))
    if words.value <= 0:
        return None
    out = np.zeros(words.value, dtype=np.uint64)
    _check("mlp_phase_cycles", load().mlp_phase_cycles(ctx.handle, out.ctypes.data, words.value,
                                                       ctypes.byref(words)))
    return out.astype(np.int64).reshape(-1, 2, 16)


def mlp_status_string(status: int) -> str:
    return load().mlp_status_string(status).decode()


# --- deeper networks (L hidden layers) ------------------------------------------

def mlp_deep_param_count(d_in: int, hidden: int, layers: int) -> int:
    return int(load().mlp_deep_param_count(d_in, hidden, layers))


class DeepContext:
    """A deep-net context bound to caller-owned parameters and workspace."""

    def __init__(self, handle, params, workspace, hidden, layers, max_batch):
        self.handle = handle
        self.params, self.workspace = params, workspace
        self.hidden, self.layers, self.max_batch = hidden, layers, max_batch

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and _lib is not None:
            _lib.mlp_deep_destroy(h)


def mlp_deep_init(params: torch.Tensor, hidden: int, layers: int, max_batch: int,
                  workspace=None, stream=None) -> DeepContext:
    """params: flat fp32 [W_1 (32 x h) | W_2 .. W_L (h x h) | w_o (h)], updated in place."""
    lib = load()
    np_ = lib.mlp_deep_param_count(D_IN, hidden, layers)
    if np_ == 0:
        raise MLPError("mlp_deep_param_count", -2)
    _dev(params, "params", numel=np_)
    need = lib.mlp_deep_workspace_bytes(D_IN, hidden, layers, max_batch)
    if need == 0:
        raise MLPError("mlp_deep_workspace_bytes", -1)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=params.device)
    _dev(workspace, "workspace", dtype=torch.uint8, numel=need)
    if stream is None:
        stream = torch.cuda.current_stream(params.device).cuda_stream
    handle = _vp()
    _check("mlp_deep_init", lib.mlp_deep_init(ctypes.byref(handle), D_IN, hidden, layers, 1,
                                              max_batch, params.data_ptr(), workspace.data_ptr(),
                                              workspace.numel(), stream))
    return DeepContext(handle, params, workspace, hidden, layers, max_batch)


def mlp_deep_forward(ctx: DeepContext, X, idx=None, B=None, out=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    if out is None:
        out = torch.empty(B, dtype=torch.float32, device=X.device)
    _check("mlp_deep_forward", load().mlp_deep_forward(ctx.handle, X.data_ptr(), n_rows,
                                                       _rows(idx, B), B,
                                                       _dev(out, "Ypred", numel=B)))
    return out


def mlp_deep_backward(ctx: DeepContext, X, Y, idx=None, B=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    _dev(Y, "Y", numel=n_rows)
    dP = torch.empty_like(ctx.params)
    loss = torch.empty(1, dtype=torch.float32, device=X.device)
    _check("mlp_deep_backward", load().mlp_deep_backward(ctx.handle, X.data_ptr(), n_rows,
                                                         Y.data_ptr(), _rows(idx, B), B,
                                                         dP.data_ptr(), loss.data_ptr()))
    return dP, loss


def mlp_deep_sgd_step(ctx: DeepContext, X, Y, lr, idx=None, B=None, loss=None):
    n_rows = X.shape[0]
    B = (n_rows if idx is None else idx.numel()) if B is None else B
    _dev(X, "X", numel=n_rows * D_IN)
    _dev(Y, "Y", numel=n_rows)
    lp = _dev(loss, "loss", numel=1) if loss is not None else None
    _check("mlp_deep_sgd_step", load().mlp_deep_sgd_step(ctx.handle, X.data_ptr(), n_rows,
                                                         Y.data_ptr(), _rows(idx, B), B,
                                                         float(lr), lp))
    return loss


def mlp_deep_train_epochs(ctx: DeepContext, X, Y, batch, lr, epochs, perm=None, max_steps=-1,
                          epoch_loss=None, step_loss=None):
    n = X.shape[0]
    _dev(X, "X", numel=n * D_IN)
    _dev(Y, "Y", numel=n)
    pp = _dev(perm, "perm", dtype=torch.int32, numel=epochs * n) if perm is not None else None
    ep = _dev(epoch_loss, "epoch_loss", numel=epochs) if epoch_loss is not None else None
    steps = -(-n // batch) * epochs
    if max_steps >= 0:
        steps = min(steps, max_steps)
    sp = _dev(step_loss, "step_loss", numel=steps) if step_loss is not None else None
    _check("mlp_deep_train_epochs", load().mlp_deep_train_epochs(ctx.handle, X.data_ptr(),
                                                                 Y.data_ptr(), n, batch, float(lr),
                                                                 epochs, pp, max_steps, ep, sp))


def mlp_deep_check_errors(ctx: DeepContext) -> None:
    _check("mlp_deep_check_errors", load().mlp_deep_check_errors(ctx.handle))


def mlp_deep_profile(ctx: DeepContext, enable: bool) -> None:
    _check("mlp_deep_profile", load().mlp_deep_profile(ctx.handle, 1 if enable else 0))


def mlp_deep_last_kernel_ms(ctx: DeepContext) -> float:
    ms = _f32(0.0)
    _check("mlp_deep_last_kernel_ms", load().mlp_deep_last_kernel_ms(ctx.handle, ctypes.byref(ms)))
    return float(ms.value)
