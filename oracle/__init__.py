"""fp64 CPU oracle for mini-batch SGD on the d-h-1 ReLU/MSE network.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The HIP training
path (``paper_2606_30497_amd``) never imports it, and this package never
imports that one; the two share no code. Both consume arrays from the
``datagen`` module, which holds no training arithmetic.

The arithmetic lives in ``oracle.c`` (plain fp64 loops, paper Sec. II.A
eqs. (1)-(9) and Sec. III eqs. (11)-(19)); this file only marshals numpy
arrays into it.

Pins (tests/test_oracle_pins.py): central finite differences, the closed form
of an all-active (linear) net, a hand-worked two-sample step, the strict
ReLU'(0) = 0 convention, torch float64 autograd at the real shapes, and
invariants of the batch-size scaling.

``oracle_mt.c`` (liboracle_mt.so, OpenMP) is the same SGD with each batch cut
into 64 fixed row chunks whose partials are summed in chunk order, so its
result does not depend on the thread count; the ``mt_*`` functions marshal into
it. Pinned to the single-thread oracle (tests/test_oracle_mt.py): forward
bitwise equal, gradients and 10-step training within 1e-13.

``oracle_deep.c`` (its own library, liboracle_deep.so, sharing no code with
oracle.c) extends the same equations to L hidden layers of width h; the
``deep_*`` functions below marshal into it. Its pins
(tests/test_oracle_deep_pins.py): agreement with oracle.c at L = 1, central
finite differences, the closed form of an all-active deep (linear) net, and
torch float64 autograd.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# where the three libraries live: beside the sources, unless ORACLE_LIBDIR names
# another build of them (the tests' sanitizer run builds one with ASan/UBSan)
_LIBDIR = os.environ.get("ORACLE_LIBDIR") or _HERE
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_LIBDIR, "liboracle.so")
_DEEP_SRC = os.path.join(_HERE, "oracle_deep.c")
_DEEP_LIB = os.path.join(_LIBDIR, "liboracle_deep.so")
_MT_SRC = os.path.join(_HERE, "oracle_mt.c")
_MT_LIB = os.path.join(_LIBDIR, "liboracle_mt.so")
_lib = None
_deep_lib = None
_mt_lib = None

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")


def _gcc(src, lib, extra=(), cc="gcc"):
    tmp = lib + ".tmp%d" % os.getpid()
    subprocess.check_call([cc, "-O2", "-std=c11", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fno-fast-math", "-Wall", *extra,
                           "-o", tmp, src, "-lm"])
    os.replace(tmp, lib)


def build(force: bool = True, out_dir: str | None = None, cc: str = "gcc",
          extra=()) -> str:
    """Compile liboracle.so, liboracle_deep.so and liboracle_mt.so (OpenMP) with
    gcc (plain -O2, no FMA contraction, no fast-math). out_dir, cc and extra
    (added flags, e.g. sanitizers) build another copy elsewhere; the copy this
    package loads is the one in ORACLE_LIBDIR, else the one beside the sources."""
    libs = [(_SRC, _LIB, ()), (_DEEP_SRC, _DEEP_LIB, ()), (_MT_SRC, _MT_LIB, ("-fopenmp",))]
    for src, lib, own in libs:
        if out_dir is not None:
            lib = os.path.join(out_dir, os.path.basename(lib))
        if force or not os.path.exists(lib):
            _gcc(src, lib, tuple(own) + tuple(extra), cc)
    return _LIB if out_dir is None else os.path.join(out_dir, os.path.basename(_LIB))


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_forward.restype = ctypes.c_int
        lib.oracle_forward.argtypes = [_f32p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                       ctypes.c_int32, ctypes.c_int32, _f64p, _f64p, _f64p]
        lib.oracle_grad.restype = ctypes.c_int
        lib.oracle_grad.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_int32, ctypes.c_int32, _f64p, _f64p, _f64p, _f64p,
                                    ctypes.POINTER(ctypes.c_double), ctypes.c_void_p,
                                    ctypes.c_void_p]
        lib.oracle_train.restype = ctypes.c_int
        lib.oracle_train.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                     _f64p, _f64p, ctypes.c_int64, ctypes.c_double,
                                     ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.POINTER(ctypes.c_int64)]
        _lib = lib
    return _lib


def _load_deep():
    global _deep_lib
    if _deep_lib is None:
        if not os.path.exists(_DEEP_LIB):
            _gcc(_DEEP_SRC, _DEEP_LIB)
        lib = ctypes.CDLL(_DEEP_LIB)
        lib.oracle_deep_param_count.restype = ctypes.c_int64
        lib.oracle_deep_param_count.argtypes = [ctypes.c_int32] * 3
        lib.oracle_deep_forward.restype = ctypes.c_int
        lib.oracle_deep_forward.argtypes = [_f32p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _f64p,
                                            _f64p]
        lib.oracle_deep_grad.restype = ctypes.c_int
        lib.oracle_deep_grad.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_void_p,
                                         ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, _f64p, _f64p,
                                         ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double)]
        lib.oracle_deep_train.restype = ctypes.c_int
        lib.oracle_deep_train.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_int32, _f64p, ctypes.c_int64,
                                          ctypes.c_double, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_int64)]
        _deep_lib = lib
    return _deep_lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _idx(idx):
    return None if idx is None else np.ascontiguousarray(idx, dtype=np.int32)


def forward(X, W1, W2, idx=None, nb=None):
    """Ypred (fp64) for rows ``idx`` of X (all rows when idx is None)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    W1 = np.ascontiguousarray(W1, dtype=np.float64)
    W2 = np.ascontiguousarray(np.reshape(W2, -1), dtype=np.float64)
    idx = _idx(idx)
    d, h = W1.shape
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    out = np.empty(nb, dtype=np.float64)
    rc = _load().oracle_forward(X, X.shape[0], _ptr(idx), nb, d, h, W1, W2, out)
    if rc != 0:
        raise ValueError("oracle_forward failed: %d" % rc)
    return out


def grad(X, Y, W1, W2, idx=None, nb=None, want_z=False):
    """Gradients of the batch MSE: returns (dW1 [d,h], dW2 [h], loss[, z, zabs])."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    W1 = np.ascontiguousarray(W1, dtype=np.float64)
    W2 = np.ascontiguousarray(np.reshape(W2, -1), dtype=np.float64)
    idx = _idx(idx)
    d, h = W1.shape
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    dW1 = np.empty((d, h), dtype=np.float64)
    dW2 = np.empty(h, dtype=np.float64)
    loss = ctypes.c_double(0.0)
    z = zabs = None
    if want_z:
        z = np.empty((nb, h), dtype=np.float64)
        zabs = np.empty((nb, h), dtype=np.float64)
    rc = _load().oracle_grad(X, Y, X.shape[0], _ptr(idx), nb, d, h, W1, W2, dW1, dW2,
                             ctypes.byref(loss), _ptr(z), _ptr(zabs))
    if rc != 0:
        raise ValueError("oracle_grad failed: %d" % rc)
    if want_z:
        return dW1, dW2, loss.value, z, zabs
    return dW1, dW2, loss.value


def train(X, Y, W1, W2, batch, lr, epochs, perm=None, max_steps=-1):
    """Mini-batch SGD in fp64. Returns dict(W1, W2, step_loss, epoch_loss, steps)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    W1 = np.array(W1, dtype=np.float64, order="C", copy=True)
    W2 = np.array(np.reshape(W2, -1), dtype=np.float64, copy=True)
    n = X.shape[0]
    d, h = W1.shape
    if perm is not None:
        perm = np.ascontiguousarray(perm, dtype=np.int32)
        if perm.shape != (epochs, n):
            raise ValueError("perm must be [epochs, n]")
    spe = -(-n // batch)
    total = spe * epochs if max_steps < 0 else min(max_steps, spe * epochs)
    step_loss = np.zeros(max(total, 1), dtype=np.float64)
    epoch_loss = np.zeros(max(epochs, 1), dtype=np.float64)
    steps = ctypes.c_int64(0)
    rc = _load().oracle_train(X, Y, n, d, h, W1, W2, batch, float(lr), epochs, _ptr(perm),
                              max_steps, _ptr(step_loss), _ptr(epoch_loss), ctypes.byref(steps))
    if rc != 0:
        raise ValueError("oracle_train failed: %d" % rc)
    return dict(W1=W1, W2=W2, step_loss=step_loss[:steps.value],
                epoch_loss=epoch_loss[:epochs], steps=steps.value)


# --- the same SGD on several host cores (oracle_mt.c) ------------------------------

def _load_mt():
    global _mt_lib
    if _mt_lib is None:
        if not os.path.exists(_MT_LIB):
            _gcc(_MT_SRC, _MT_LIB, ("-fopenmp",))
        lib = ctypes.CDLL(_MT_LIB)
        lib.oracle_mt_threads.restype = ctypes.c_int
        lib.oracle_mt_threads.argtypes = []
        lib.oracle_mt_set_threads.restype = ctypes.c_int
        lib.oracle_mt_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_mt_forward.restype = ctypes.c_int
        lib.oracle_mt_forward.argtypes = [_f32p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_int32, ctypes.c_int32, _f64p, _f64p, _f64p]
        lib.oracle_mt_grad.restype = ctypes.c_int
        lib.oracle_mt_grad.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_void_p,
                                       ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _f64p,
                                       _f64p, _f64p, _f64p, ctypes.POINTER(ctypes.c_double)]
        lib.oracle_mt_train.restype = ctypes.c_int
        lib.oracle_mt_train.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_int32, _f64p, _f64p, ctypes.c_int64,
                                        ctypes.c_double, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.POINTER(ctypes.c_int64)]
        _mt_lib = lib
    return _mt_lib


def mt_threads():
    """Threads the multi-core oracle runs on (OMP_NUM_THREADS, else every core
    the process may use)."""
    return int(_load_mt().oracle_mt_threads())


def mt_set_threads(n):
    """Run the following multi-core oracle calls on n threads; returns the
    previous count."""
    return int(_load_mt().oracle_mt_set_threads(int(n)))


def mt_forward(X, W1, W2, idx=None, nb=None):
    """forward() on every host core: the same values, row by row."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    W1 = np.ascontiguousarray(W1, dtype=np.float64)
    W2 = np.ascontiguousarray(np.reshape(W2, -1), dtype=np.float64)
    idx = _idx(idx)
    d, h = W1.shape
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    out = np.empty(nb, dtype=np.float64)
    rc = _load_mt().oracle_mt_forward(X, X.shape[0], _ptr(idx), nb, d, h, W1, W2, out)
    if rc != 0:
        raise ValueError("oracle_mt_forward failed: %d" % rc)
    return out


def mt_grad(X, Y, W1, W2, idx=None, nb=None):
    """grad() with each batch cut into 64 row chunks summed in chunk order:
    returns (dW1, dW2, loss)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    W1 = np.ascontiguousarray(W1, dtype=np.float64)
    W2 = np.ascontiguousarray(np.reshape(W2, -1), dtype=np.float64)
    idx = _idx(idx)
    d, h = W1.shape
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    dW1 = np.empty((d, h), dtype=np.float64)
    dW2 = np.empty(h, dtype=np.float64)
    loss = ctypes.c_double(0.0)
    rc = _load_mt().oracle_mt_grad(X, Y, X.shape[0], _ptr(idx), nb, d, h, W1, W2, dW1, dW2,
                                   ctypes.byref(loss))
    if rc != 0:
        raise ValueError("oracle_mt_grad failed: %d" % rc)
    return dW1, dW2, loss.value


def mt_train(X, Y, W1, W2, batch, lr, epochs, perm=None, max_steps=-1):
    """train() with chunked batch gradients on every host core; same outputs."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    W1 = np.array(W1, dtype=np.float64, order="C", copy=True)
    W2 = np.array(np.reshape(W2, -1), dtype=np.float64, copy=True)
    n = X.shape[0]
    d, h = W1.shape
    if perm is not None:
        perm = np.ascontiguousarray(perm, dtype=np.int32)
        if perm.shape != (epochs, n):
            raise ValueError("perm must be [epochs, n]")
    spe = -(-n // batch)
    total = spe * epochs if max_steps < 0 else min(max_steps, spe * epochs)
    step_loss = np.zeros(max(total, 1), dtype=np.float64)
    epoch_loss = np.zeros(max(epochs, 1), dtype=np.float64)
    steps = ctypes.c_int64(0)
    rc = _load_mt().oracle_mt_train(X, Y, n, d, h, W1, W2, batch, float(lr), epochs,
                                    _ptr(perm), max_steps, _ptr(step_loss), _ptr(epoch_loss),
                                    ctypes.byref(steps))
    if rc != 0:
        raise ValueError("oracle_mt_train failed: %d" % rc)
    return dict(W1=W1, W2=W2, step_loss=step_loss[:steps.value],
                epoch_loss=epoch_loss[:epochs], steps=steps.value)


# --- L hidden layers (oracle_deep.c) -------------------------------------------

def deep_param_count(d, h, L):
    return int(_load_deep().oracle_deep_param_count(d, h, L))


def deep_split(P, d, h, L):
    """Views of a flat parameter array: ([W_1, ..., W_L], w_o)."""
    P = np.asarray(P)
    Ws, off = [], 0
    for l in range(L):
        K = d if l == 0 else h
        Ws.append(P[off:off + K * h].reshape(K, h))
        off += K * h
    return Ws, P[off:off + h]


def deep_forward(X, P, d, h, L, idx=None, nb=None):
    """Ypred (fp64) of the L-hidden-layer net for rows ``idx`` of X."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    P = np.ascontiguousarray(P, dtype=np.float64)
    idx = _idx(idx)
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    out = np.empty(nb, dtype=np.float64)
    rc = _load_deep().oracle_deep_forward(X, X.shape[0], _ptr(idx), nb, d, h, L, P, out)
    if rc != 0:
        raise ValueError("oracle_deep_forward failed: %d" % rc)
    return out


def deep_grad(X, Y, P, d, h, L, idx=None, nb=None):
    """Gradients of the batch MSE: returns (dP flat fp64, loss, margin), margin =
    the smallest |Z| / sum |terms| over every pre-activation of the batch."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    P = np.ascontiguousarray(P, dtype=np.float64)
    idx = _idx(idx)
    if nb is None:
        nb = X.shape[0] if idx is None else idx.shape[0]
    dP = np.empty_like(P)
    loss = ctypes.c_double(0.0)
    margin = ctypes.c_double(0.0)
    rc = _load_deep().oracle_deep_grad(X, Y, X.shape[0], _ptr(idx), nb, d, h, L, P, dP,
                                       ctypes.byref(loss), ctypes.byref(margin))
    if rc != 0:
        raise ValueError("oracle_deep_grad failed: %d" % rc)
    return dP, loss.value, margin.value


def deep_train(X, Y, P, d, h, L, batch, lr, epochs, perm=None, max_steps=-1):
    """Mini-batch SGD of the L-hidden-layer net in fp64. Returns dict(P,
    step_loss, epoch_loss, steps)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    Y = np.ascontiguousarray(np.reshape(Y, -1), dtype=np.float32)
    P = np.array(P, dtype=np.float64, order="C", copy=True)
    n = X.shape[0]
    if perm is not None:
        perm = np.ascontiguousarray(perm, dtype=np.int32)
        if perm.shape != (epochs, n):
            raise ValueError("perm must be [epochs, n]")
    spe = -(-n // batch)
    total = spe * epochs if max_steps < 0 else min(max_steps, spe * epochs)
    step_loss = np.zeros(max(total, 1), dtype=np.float64)
    epoch_loss = np.zeros(max(epochs, 1), dtype=np.float64)
    steps = ctypes.c_int64(0)
    rc = _load_deep().oracle_deep_train(X, Y, n, d, h, L, P, batch, float(lr), epochs,
                                        _ptr(perm), max_steps, _ptr(step_loss),
                                        _ptr(epoch_loss), ctypes.byref(steps))
    if rc != 0:
        raise ValueError("oracle_deep_train failed: %d" % rc)
    return dict(P=P, step_loss=step_loss[:steps.value], epoch_loss=epoch_loss[:epochs],
                steps=steps.value)


class swapped_deep_library:
    """Points the deep_* functions at another build of oracle_deep.c (mutation
    tests only)."""

    def __init__(self, path):
        self.path = path
        self.saved = None

    def __enter__(self):
        global _deep_lib, _DEEP_LIB
        self.saved = (_deep_lib, _DEEP_LIB)
        _deep_lib, _DEEP_LIB = None, self.path
        _load_deep()
        return self

    def __exit__(self, *exc):
        global _deep_lib, _DEEP_LIB
        _deep_lib, _DEEP_LIB = self.saved
        return False


class swapped_library:
    """Context manager that points this module at another build of oracle.c.

    Used only by the mutation tests, which compile deliberately broken copies
    of the oracle and check that the pins reject each of them."""

    def __init__(self, path):
        self.path = path
        self.saved = None

    def __enter__(self):
        global _lib, _LIB
        self.saved = (_lib, _LIB)
        _lib, _LIB = None, self.path
        _load()
        return self

    def __exit__(self, *exc):
        global _lib, _LIB
        _lib, _LIB = self.saved
        return False
