"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point include/mlp.h declares, sizes its workspace, and rejects bad
arguments before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mlp.h")


def _lib():
    from paper_2606_30497_amd import mlp
    if not os.path.exists(mlp.library_path()):
        pytest.skip("libmlp.so not built")
    return mlp.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mlp_[a-z_]+)\s*\(", text)))


def test_header_declares_the_five_calls():
    names = declared_functions()
    for f in ("mlp_init", "mlp_forward", "mlp_backward", "mlp_sgd_step", "mlp_train_epochs"):
        assert f in names


def test_every_declared_symbol_is_exported():
    lib = _lib()
    from paper_2606_30497_amd import mlp
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in mlp.EXPORTS, name


def test_workspace_bytes():
    lib = _lib()
    for h in (32, 64, 128, 256, 512, 1024):
        b = lib.mlp_workspace_bytes(32, h, 4096)
        assert b > 0 and b % 256 == 0
        assert lib.mlp_workspace_bytes(32, h, 1 << 20) >= b
    assert lib.mlp_workspace_bytes(32, 100, 64) == 0
    assert lib.mlp_workspace_bytes(16, 256, 64) == 0
    assert lib.mlp_workspace_bytes(32, 256, 0) == 0
    assert lib.mlp_workspace_bytes(32, 256, (1 << 20) + 1) == 0


def test_strategy_workspace_bytes():
    lib = _lib()
    for h in (32, 256, 1024):
        for strat in (2, 3):   # OPTIMIZED, BASELINE: intermediates of one step
            b = lib.mlp_strategy_workspace_bytes(32, h, 256, strat)
            assert b % 256 == 0 and b >= 4 * 256 * (6 * h + 68)
            assert lib.mlp_strategy_workspace_bytes(32, h, 4096, strat) > b
        for strat in (0, 1):   # FUSED, TILE need none
            assert lib.mlp_strategy_workspace_bytes(32, h, 256, strat) == 0
    assert lib.mlp_strategy_workspace_bytes(32, 256, 256, 4) == 0
    assert lib.mlp_strategy_workspace_bytes(32, 100, 256, 2) == 0
    assert lib.mlp_strategy_workspace_bytes(32, 256, 0, 2) == 0


def test_deep_sizes_and_checks():
    lib = _lib()
    assert lib.mlp_deep_param_count(32, 256, 1) == 8448
    assert lib.mlp_deep_param_count(32, 256, 3) == 32 * 256 + 2 * 256 * 256 + 256
    for bad in ((32, 100, 2), (32, 32, 2), (16, 256, 2), (32, 256, 0), (32, 256, 9), (32, 2048, 2)):
        assert lib.mlp_deep_param_count(*bad) == 0
        assert lib.mlp_deep_workspace_bytes(*bad, 64) == 0
    b = lib.mlp_deep_workspace_bytes(32, 256, 3, 4096)
    assert b >= 4 * (3 * 4096 * 256) and b % 256 == 0
    assert lib.mlp_deep_workspace_bytes(32, 256, 3, 0) == 0
    h = ctypes.c_void_p()
    fake = ctypes.c_void_p(256)
    assert lib.mlp_deep_init(None, 32, 256, 2, 1, 64, fake, fake, 1 << 30, None) == -1
    assert lib.mlp_deep_init(ctypes.byref(h), 32, 256, 2, 2, 64, fake, fake, 1 << 30, None) == -2
    assert lib.mlp_deep_init(ctypes.byref(h), 32, 256, 2, 1, 64, fake, fake, 100, None) == -3
    assert h.value is None
    assert lib.mlp_deep_forward(None, fake, 10, None, 10, fake) == -1
    assert lib.mlp_deep_check_errors(None) == -1


def declared_statuses():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return {name: int(v) for name, v in re.findall(r"\b(MLP_(?:OK|ERR_[A-Z_]+))\s*=\s*(-?\d+)", text)}


def test_status_strings():
    """Every status the header declares has a message in the library and its
    name in the binding."""
    lib = _lib()
    from paper_2606_30497_amd import mlp
    codes = declared_statuses()
    assert codes["MLP_OK"] == 0 and codes["MLP_ERR_NONFINITE"] == -5
    assert len(set(codes.values())) == len(codes)
    for name, v in codes.items():
        assert lib.mlp_status_string(v) != b"unknown status", name
        assert mlp.STATUS[v] == name
    assert lib.mlp_status_string(-99) == b"unknown status"


def test_init_rejects_bad_arguments_without_device():
    lib = _lib()
    h = ctypes.c_void_p()
    fake = ctypes.c_void_p(256)      # never dereferenced: validation fails first
    ws = lib.mlp_workspace_bytes(32, 256, 64)
    # null out-pointer / weights / workspace
    assert lib.mlp_init(None, 32, 256, 1, 64, fake, fake, fake, ws, None) == -1
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 1, 64, None, fake, fake, ws, None) == -1
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 1, 64, fake, fake, None, ws, None) == -1
    # unsupported shapes
    assert lib.mlp_init(ctypes.byref(h), 16, 256, 1, 64, fake, fake, fake, ws, None) == -2
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 2, 64, fake, fake, fake, ws, None) == -2
    assert lib.mlp_init(ctypes.byref(h), 32, 100, 1, 64, fake, fake, fake, ws, None) == -2
    # batch limits, workspace size and alignment
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 1, 0, fake, fake, fake, ws, None) == -1
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 1, 64, fake, fake, fake, ws - 1, None) == -3
    assert lib.mlp_init(ctypes.byref(h), 32, 256, 1, 64, fake, fake, ctypes.c_void_p(260), ws,
                        None) == -3
    assert h.value is None


def test_null_context_is_rejected():
    lib = _lib()
    fake = ctypes.c_void_p(256)
    assert lib.mlp_forward(None, fake, 10, None, 10, fake) == -1
    assert lib.mlp_backward(None, fake, 10, fake, None, 10, fake, fake, None) == -1
    assert lib.mlp_sgd_step(None, fake, 10, fake, None, 10, 0.1, None) == -1
    assert lib.mlp_train_epochs(None, fake, fake, 10, 2, 0.1, 1, None, -1, None, None) == -1
    assert lib.mlp_check_errors(None) == -1
    assert lib.mlp_profile(None, 1) == -1
    assert lib.mlp_set_strategy(None, 0, None, 0) == -1
    lib.mlp_destroy(None)


def test_static_entry_rejects_before_any_hip_call():
    """mlp_train_epochs_static checks its arguments before its first HIP call, so
    these run without a GPU (the pointers are never dereferenced)."""
    lib = _lib()
    f = ctypes.c_void_p(256)

    def call(h=256, n=64, batch=64, lr=0.01, epochs=1, max_steps=-1, w1=f):
        return lib.mlp_train_epochs_static(h, w1, f, f, f, n, batch, lr, epochs, None, max_steps,
                                           None, None, None, None)

    assert call(h=512) == -3 and call(h=1024) == -3       # beyond the 16 MiB scratch
    assert call(h=48) == -2 and call(h=2048) == -2        # unsupported widths
    assert call(batch=0) == -1 and call(batch=(1 << 20) + 1) == -1
    assert call(n=0) == -1 and call(epochs=0) == -1 and call(max_steps=-2) == -1
    assert call(lr=float("nan")) == -1 and call(lr=float("inf")) == -1
    assert call(w1=None) == -1
