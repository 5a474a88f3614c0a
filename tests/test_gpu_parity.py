"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerances (normwise relative error unless stated):
  - per-step gradients dW1, dW2: <= 1e-4, after ReLU-kink alignment of dW1;
  - forward outputs: <= 1e-5; batch loss: 1e-5 relative plus the fp32 forward
    rounding term of tests/parity.py:loss_tolerance (matters where Ypred ~ Y);
  - weights and per-step losses after 10 SGD steps: <= 1e-3, on every
    workload, and so is the weight change W10 - W0 (the meaningful check, since
    lr * dW is small against W);
  - the full-dataset MSE at the weights after those 10 steps, the GPU's own
    forward pass over every row (mlp_forward) against the oracle's forward at
    the oracle's weights: <= 1e-3 relative;
  - gradients at trained weights (after 10 steps of the largest workload): the
    per-step bar, 1e-4.
Every weight and gradient check holds both the normwise and the largest
elementwise error (tests/parity.py:check) to its bar.
"""
import numpy as np
import pytest
import torch

import datagen
import oracle
from tests.parity import align_kinks, check, loss_tolerance, rel

pytestmark = pytest.mark.gpu

H_ALL = (32, 64, 128, 256, 512, 1024)


@pytest.fixture(scope="module")
def mlp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_30497_amd import mlp as m
    m.load(require_built=True)
    return m


def _to(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def _ctx(mlp, W1, W2, max_batch, strategy=None):
    w1 = _to(W1.astype(np.float32))
    w2 = _to(np.reshape(W2, -1).astype(np.float32))
    ctx = mlp.mlp_init(w1, w2, max_batch)
    if strategy is not None:
        mlp.mlp_set_strategy(ctx, strategy)
    return ctx, w1, w2


def _rows(rng, n, B):
    return rng.integers(0, n, size=B).astype(np.int32)


# --- forward -------------------------------------------------------------------

@pytest.mark.parametrize("h", H_ALL)
def test_forward_matches_oracle(mlp, h):
    rng = np.random.default_rng(h)
    d = datagen.make_data(3001, h, seed=100 + h, with_perm=False)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, 64)
    X = _to(d.X)
    idx = _rows(rng, 3001, 2777)
    yp = mlp.mlp_forward(ctx, X, _to(idx)).cpu().numpy()
    ref = oracle.forward(d.X, d.W1, d.W2, idx=idx)
    assert rel(yp, ref) < 1e-5
    yp_all = mlp.mlp_forward(ctx, X).cpu().numpy()
    assert rel(yp_all, oracle.forward(d.X, d.W1, d.W2)) < 1e-5
    mlp.mlp_check_errors(ctx)


@pytest.mark.parametrize("h", H_ALL)
@pytest.mark.parametrize("B", [1, 15, 16, 17, 1000])
def test_forward_ragged_batches(mlp, h, B):
    d = datagen.make_data(1200, h, seed=110 + h, with_perm=False)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, 64)
    idx = np.random.default_rng(B).integers(0, 1200, size=B).astype(np.int32)
    out = torch.full((B + 40,), 7.0, device="cuda")        # guard words past B stay untouched
    mlp.mlp_forward(ctx, _to(d.X), _to(idx), B=B, out=out)
    got = out.cpu().numpy()
    assert rel(got[:B], oracle.forward(d.X, d.W1, d.W2, idx=idx)) < 1e-5
    assert np.all(got[B:] == 7.0)
    mlp.mlp_check_errors(ctx)


@pytest.mark.parametrize("k", [3, 4])
def test_forward_full_dataset_sampled(mlp, k):
    """mlp_forward over every row of the 1M-row (h = 1024) and 10M-row (h = 256)
    datasets, in the launch shape of the forward benchmark; 20,000 sampled outputs
    against the oracle, and every output finite."""
    w, d = _workload_data(k)
    print("workload", w.name, flush=True)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, 64)
    X = _to(d.X)
    out = mlp.mlp_forward(ctx, X)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    assert bool(torch.isfinite(out).all())
    sample = np.random.default_rng(k).integers(0, w.n, size=20000).astype(np.int64)
    sample[:2] = [0, w.n - 1]
    got = out.cpu().numpy()[sample]
    ref = oracle.forward(d.X, d.W1, d.W2, idx=sample.astype(np.int32))
    assert rel(got, ref) < 1e-5


@pytest.mark.parametrize("h", [32, 64])
def test_forward_full_dataset_sampled_narrow(mlp, h):
    """The narrow nets over all 10M rows of the largest workload's X in the
    forward benchmark's launch shape (at h = 32 two row tiles per wave per
    iteration): 20,000 sampled outputs against the oracle, every output finite."""
    w, d = _workload_data(4)
    net = datagen.make_data(1, h, seed=2000 + h, with_perm=False)
    ctx, _, _ = _ctx(mlp, net.W1, net.W2, 64)
    out = mlp.mlp_forward(ctx, _to(d.X))
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    assert bool(torch.isfinite(out).all())
    sample = np.random.default_rng(h).integers(0, w.n, size=20000).astype(np.int64)
    sample[:2] = [0, w.n - 1]
    got = out.cpu().numpy()[sample]
    ref = oracle.forward(d.X, net.W1, net.W2, idx=sample.astype(np.int32))
    assert rel(got, ref) < 1e-5


# --- per-step gradients ----------------------------------------------------------

def _check_grad(mlp, h, B, n=5000, seed=0, idx_none=False, strategy=None):
    rng = np.random.default_rng(seed)
    d = datagen.make_data(n, h, seed=200 + h + B, with_perm=False)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, max(B, 1), strategy)
    idx = None if idx_none else _rows(rng, n, B)
    dW1, dW2, loss = mlp.mlp_backward(ctx, _to(d.X), _to(d.Y), None if idx is None else _to(idx),
                                      B=B)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    g1, g2, gl = dW1.cpu().numpy(), dW2.cpu().numpy(), float(loss.cpu()[0])
    W1, W2 = d.W1.astype(np.float64), d.W2.astype(np.float64)
    r1, r2, rL, z, zabs = oracle.grad(d.X, d.Y, W1, W2, idx=idx, nb=B, want_z=True)
    yp = oracle.forward(d.X, W1, W2, idx=idx, nb=B)
    r1a, n_amb, flips = align_kinks(g1, r1, d.X, d.Y, W1, W2, idx, z, zabs, yp)
    print("kink entries %d, flips accepted %d" % (n_amb, flips))
    e1, _ = check("dW1", g1, r1a, 1e-4)
    e2, _ = check("dW2", g2, r2, 1e-4)
    assert abs(gl - rL) <= loss_tolerance(rL, z, zabs, W2)
    return e1, e2


@pytest.mark.parametrize("h", H_ALL)
@pytest.mark.parametrize("B", [1, 7, 64, 160, 1000])
def test_backward_small_batches(mlp, h, B):
    _check_grad(mlp, h, B, seed=B)


@pytest.mark.parametrize("h,B", [(256, 4096), (256, 1664), (256, 576), (1024, 1024),
                                 (1024, 576), (256, 256), (256, 64)])
def test_backward_workload_batches(mlp, h, B):
    _check_grad(mlp, h, B, n=20000, seed=B)


def test_backward_identity_rows(mlp):
    _check_grad(mlp, 256, 333, n=333, idx_none=True)


# --- worked examples embedded in 32-h-1 by zero padding ---------------------------

def _embed(X, W1, W2, h):
    Xp = np.zeros((X.shape[0], 32), np.float32)
    Xp[:, :X.shape[1]] = X
    W1p = np.zeros((32, h), np.float32)
    W1p[:W1.shape[0], :W1.shape[1]] = W1
    W2p = np.zeros(h, np.float32)
    W2p[:W2.shape[0]] = W2
    return Xp, W1p, W2p


@pytest.mark.parametrize("h", [32, 256, 1024])
def test_worked_two_sample_step_embedded(mlp, h):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_two_sample.json")))
    X, W1, W2 = _embed(np.array(g["X"], np.float32), np.array(g["W1"]), np.array(g["W2"]), h)
    Y = np.array(g["Y"], np.float32)
    ctx, w1, w2 = _ctx(mlp, W1, W2, 2)
    dW1, dW2, loss = mlp.mlp_backward(ctx, _to(X), _to(Y))
    dW1, dW2 = dW1.cpu().numpy(), dW2.cpu().numpy()
    exp1 = np.zeros((32, h)); exp1[:2, :2] = g["dW1"]
    exp2 = np.zeros(h); exp2[:2] = g["dW2"]
    assert np.array_equal(dW1, exp1) and np.array_equal(dW2, exp2)
    assert float(loss.cpu()[0]) == g["loss"]
    mlp.mlp_sgd_step(ctx, _to(X), _to(Y), g["lr"])
    np.testing.assert_allclose(w1.cpu().numpy()[:2, :2], g["W1_next"], atol=1e-6)
    np.testing.assert_allclose(w2.cpu().numpy()[:2], g["W2_next"], atol=1e-6)
    assert np.all(w1.cpu().numpy()[2:, :] == 0) and np.all(w1.cpu().numpy()[:, 2:] == 0)
    assert np.all(w2.cpu().numpy()[2:] == 0)


def test_relu_zero_embedded(mlp):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "relu_zero.json")))
    X, W1, W2 = _embed(np.array(g["X"], np.float32), np.array(g["W1"]), np.array(g["W2"]), 256)
    ctx, _, _ = _ctx(mlp, W1, W2, 1)
    dW1, dW2, loss = mlp.mlp_backward(ctx, _to(X), _to(np.array(g["Y"], np.float32)))
    assert torch.all(dW1 == 0) and torch.all(dW2 == 0)
    assert float(loss.cpu()[0]) == g["loss"]


# --- training ------------------------------------------------------------------

_DATA = {}


def _workload_data(k):
    if k not in _DATA:
        _DATA.clear()
        w = datagen.WORKLOADS[k]
        d = datagen.make_workload(w)
        _DATA[k] = (w, d)
    return _DATA[k]


def _train_gpu(mlp, d, batch, lr, epochs, max_steps=-1, perm=None, strategy=None):
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, batch, strategy)
    n = d.X.shape[0]
    spe = -(-n // batch)
    steps = spe * epochs if max_steps < 0 else min(max_steps, spe * epochs)
    el = torch.zeros(epochs, dtype=torch.float32, device="cuda")
    sl = torch.zeros(steps, dtype=torch.float32, device="cuda")
    p = None if perm is None else _to(perm)
    mlp.mlp_train_epochs(ctx, _to(d.X), _to(d.Y), batch, lr, epochs, perm=p, max_steps=max_steps,
                         epoch_loss=el, step_loss=sl)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    return w1.cpu().numpy(), w2.cpu().numpy(), sl.cpu().numpy(), el.cpu().numpy()


@pytest.mark.parametrize("k", range(5))
def test_train_ten_steps_full_workload(mlp, k):
    w, d = _workload_data(k)
    print("workload", w.name, flush=True)
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, w.batch)
    sl = torch.zeros(10, dtype=torch.float32, device="cuda")
    X, Y = _to(d.X), _to(d.Y)
    perm = None if d.perm is None else _to(d.perm)
    mlp.mlp_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=perm, max_steps=10,
                         step_loss=sl)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    g1, g2, gsl = w1.cpu().numpy(), w2.cpu().numpy(), sl.cpu().numpy()
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, w.batch, w.lr, w.epochs, perm=d.perm, max_steps=10)
    W10, W20 = d.W1.astype(np.float64), d.W2.astype(np.float64)
    check("W1", g1, ref["W1"], 1e-3)
    check("W2", g2, ref["W2"], 1e-3)
    check("W1 - W1_0", g1 - W10, ref["W1"] - W10, 1e-3)
    check("W2 - W2_0", g2 - W20, ref["W2"] - W20, 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * np.abs(ref["step_loss"]))
    # full-dataset MSE at the trained weights: the GPU's forward pass over every
    # row (eqs. 11-14) against the oracle's forward at the oracle's weights
    yp = mlp.mlp_forward(ctx, X).cpu().numpy().astype(np.float64)
    mse_gpu = float(np.mean((yp - d.Y) ** 2))
    mse_ref = float(np.mean((oracle.mt_forward(d.X, ref["W1"], ref["W2"]) - d.Y) ** 2))
    print("full-dataset MSE at W10: gpu %.6e oracle %.6e rel %.3e" %
          (mse_gpu, mse_ref, abs(mse_gpu - mse_ref) / mse_ref))
    assert abs(mse_gpu - mse_ref) <= 1e-3 * mse_ref


def test_gradients_at_trained_weights(mlp):
    """Per-step gradients of the largest workload at the weights its first 10 SGD
    steps on the GPU reached (not only at the initial weights): a full batch of
    4096 rows and the 1664-row tail size, each against the oracle at the same
    fp32 weights, kink-aligned, <= 1e-4."""
    w, d = _workload_data(4)
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, w.batch)
    X, Y = _to(d.X), _to(d.Y)
    mlp.mlp_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=_to(d.perm), max_steps=10)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    W1t = w1.cpu().numpy().astype(np.float64)
    W2t = w2.cpu().numpy().astype(np.float64)
    rng = np.random.default_rng(5)
    for B in (4096, 1664):
        idx = rng.integers(0, w.n, size=B).astype(np.int32)
        dW1, dW2, loss = mlp.mlp_backward(ctx, X, Y, _to(idx), B=B)
        torch.cuda.synchronize()
        mlp.mlp_check_errors(ctx)
        g1, g2, gl = dW1.cpu().numpy(), dW2.cpu().numpy(), float(loss.cpu()[0])
        r1, r2, rL, z, zabs = oracle.grad(d.X, d.Y, W1t, W2t, idx=idx, want_z=True)
        yp = oracle.forward(d.X, W1t, W2t, idx=idx)
        r1a, n_amb, flips = align_kinks(g1, r1, d.X, d.Y, W1t, W2t, idx, z, zabs, yp)
        print("B %d: kink entries %d, flips accepted %d" % (B, n_amb, flips))
        check("dW1 (trained, B=%d)" % B, g1, r1a, 1e-4)
        check("dW2 (trained, B=%d)" % B, g2, r2, 1e-4)
        assert abs(gl - rL) <= loss_tolerance(rL, z, zabs, W2t)


@pytest.mark.parametrize("w", datagen.SWEEP, ids=lambda w: w.name)
def test_sweep_workload_steps(mlp, w):
    """Hidden-width sweep (Table II sizes): the first 20 steps (two epochs, a fresh
    permutation each) match the oracle's weights, weight change and step losses."""
    d = datagen.make_workload(w)
    g1, g2, gsl, gel = _train_gpu(mlp, d, w.batch, w.lr, w.epochs, max_steps=20, perm=d.perm)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, w.batch, w.lr, w.epochs, perm=d.perm, max_steps=20)
    W10 = d.W1.astype(np.float64)
    check("W1 - W1_0", g1 - W10, ref["W1"] - W10, 1e-3)
    check("W2 - W2_0", g2 - d.W2, ref["W2"] - d.W2.astype(np.float64), 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * np.abs(ref["step_loss"]))
    assert np.all(np.abs(gel[:2] - ref["epoch_loss"][:2]) <= 1e-3 * ref["epoch_loss"][:2])


def test_train_epochs_with_tail_and_shuffle(mlp):
    n, h, B, E, lr = 1000, 256, 64, 3, 0.01
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=77)
    g1, g2, gsl, gel = _train_gpu(mlp, d, B, lr, E, perm=d.perm)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, lr, E, perm=d.perm)
    assert len(gsl) == ref["steps"] == 48
    check("W1 - W1_0", g1 - d.W1, ref["W1"] - d.W1.astype(np.float64), 1e-3)
    check("W2 - W2_0", g2 - d.W2, ref["W2"] - d.W2.astype(np.float64), 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-3 * ref["epoch_loss"])


def test_full_first_workload_run(mlp):
    w, d = _workload_data(0)
    g1, g2, gsl, gel = _train_gpu(mlp, d, w.batch, w.lr, w.epochs, perm=d.perm)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, w.batch, w.lr, w.epochs, perm=d.perm)
    assert ref["steps"] == 80
    check("W1 - W1_0", g1 - d.W1, ref["W1"] - d.W1.astype(np.float64), 1e-3)
    check("W2 - W2_0", g2 - d.W2, ref["W2"] - d.W2.astype(np.float64), 1e-3)
    check("W2", g2, ref["W2"], 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-3 * ref["epoch_loss"])


def test_deterministic_and_prefix_consistent(mlp):
    w, d = _workload_data(1)
    a = _train_gpu(mlp, d, w.batch, w.lr, 2, perm=d.perm[:2].copy())
    b = _train_gpu(mlp, d, w.batch, w.lr, 2, perm=d.perm[:2].copy())
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    c = _train_gpu(mlp, d, w.batch, w.lr, 2, max_steps=10, perm=d.perm[:2].copy())
    assert np.array_equal(c[2], a[2][:10])
    # epoch loss is the row-weighted mean of the step losses
    spe = w.steps_per_epoch
    nb = np.full(spe, w.batch, np.float64)
    nb[-1] = w.tail
    for e in range(2):
        exp = np.sum(a[2][e * spe:(e + 1) * spe] * nb) / w.n
        assert abs(a[3][e] - exp) <= 1e-5 * exp
    assert a[3][1] < a[3][0]


def test_identity_order_when_perm_is_null(mlp):
    w, d = _workload_data(0)
    a = _train_gpu(mlp, d, w.batch, w.lr, 2)
    b = _train_gpu(mlp, d, w.batch, w.lr, 2, perm=datagen.identity_perm(2, w.n))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# --- errors --------------------------------------------------------------------

def test_out_of_range_row_is_flagged_not_read(mlp):
    d = datagen.make_data(100, 256, seed=1, with_perm=False)
    ctx, w1, _ = _ctx(mlp, d.W1, d.W2, 64)
    idx = np.arange(64, dtype=np.int32)
    idx[5] = 100                        # one past the end: the kernel reads row 0 instead
    mlp.mlp_backward(ctx, _to(d.X), _to(d.Y), _to(idx))
    with pytest.raises(mlp.MLPError) as ei:
        mlp.mlp_check_errors(ctx)
    assert ei.value.status == -6
    mlp.mlp_check_errors(ctx)          # the flag is cleared by the check


def test_host_argument_errors_leave_weights_untouched(mlp):
    d = datagen.make_data(100, 256, seed=2, with_perm=False)
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, 64)
    before = (w1.clone(), w2.clone())
    X, Y = _to(d.X), _to(d.Y)
    lib = mlp.load()
    assert lib.mlp_sgd_step(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 65, 0.1, None) == -1
    assert lib.mlp_sgd_step(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 64,
                            float("nan"), None) == -1
    assert lib.mlp_sgd_step(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 0, 0.1, None) == -1
    assert lib.mlp_train_epochs(ctx.handle, X.data_ptr(), Y.data_ptr(), 100, 65, 0.1, 1, None, -1,
                                None, None) == -1
    assert lib.mlp_train_epochs(ctx.handle, X.data_ptr(), Y.data_ptr(), 100, 64, 0.1, 0, None, -1,
                                None, None) == -1
    assert lib.mlp_backward(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 101, None, None,
                            None) == -1
    torch.cuda.synchronize()
    assert torch.equal(before[0], w1) and torch.equal(before[1], w2)


# --- every plan of the persistent trainer, both paths, the coherent fallback -----

import os
import contextlib


@contextlib.contextmanager
def _env(**kv):
    old = {k: os.environ.get(k) for k in kv}
    try:
        for k, v in kv.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = str(v)
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


# The fused trainer's instantiated shapes: (groups PX, workgroups per group PR,
# rows per workgroup R, units per group U); hidden = PX * U, batch <= PR * R.
FUSED_SHAPES = [(8, 32, 128, 32), (8, 32, 64, 32), (8, 32, 32, 32), (4, 32, 16, 64),
                (1, 16, 16, 256), (8, 32, 32, 128), (8, 32, 16, 128),
                (8, 32, 16, 64), (2, 16, 16, 64), (1, 16, 16, 64), (1, 8, 32, 32),
                (4, 16, 16, 64), (2, 16, 16, 128), (4, 4, 16, 64), (8, 4, 32, 32),
                (8, 8, 32, 32)]
# Index = position in the library's shape table. A one-XCD shape with four
# workgroups of 64 owned units each, (1, 4, 16, 256), gave wrong gradient sums
# from the second SGD step on, and one run of it faulted the GPU, under the
# kernel's first ownership scheme; the cause was not found. The owner waves of
# the current kernel cap a workgroup at 16 owned units (a compile-time
# assertion), so the shape is not instantiated.


@pytest.mark.skip(reason="shape (1, 4, 16, 256) excluded: failed under the first ownership "
                         "scheme (cause not found); the current one owns at most 16 units "
                         "per workgroup, so it is not instantiated")
def test_disabled_shape_four_workgroups_one_xcd():
    pass


@pytest.mark.parametrize("inst", range(len(FUSED_SHAPES)))
def test_backward_every_fused_shape(mlp, inst):
    px, pr, r, u = FUSED_SHAPES[inst]
    h, cap = px * u, pr * r
    with _env(MLP_INST=inst):
        d = datagen.make_data(64, h, seed=4, with_perm=False)
        ctx, _, _ = _ctx(mlp, d.W1, d.W2, cap)
        wg, launches = mlp.mlp_launch_info(ctx, cap, cap, 1)
        assert (wg, launches) == (8 * pr, 1), "shape table out of step with the library"
        for B in sorted({cap, cap - 7, cap // 2 + 3, 1}):
            _check_grad(mlp, h, B, n=max(6000, cap), seed=inst * 7 + B)


@pytest.mark.parametrize("inst", range(len(FUSED_SHAPES)))
def test_train_every_fused_shape(mlp, inst):
    px, pr, r, u = FUSED_SHAPES[inst]
    h, B = px * u, pr * r
    n, E, lr = 3 * B - 5, 2, 0.005                 # a short tail batch every epoch
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=300 + inst)
    with _env(MLP_INST=inst):
        g1, g2, gsl, gel = _train_gpu(mlp, d, B, lr, E, perm=d.perm)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, lr, E, perm=d.perm)
    check("W1 - W1_0", g1 - d.W1, ref["W1"] - d.W1.astype(np.float64), 1e-3)
    check("W2 - W2_0", g2 - d.W2, ref["W2"] - d.W2.astype(np.float64), 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-3 * ref["epoch_loss"])


def test_coherent_fallback_is_bitwise_identical(mlp):
    n, h, B, E, lr = 2000, 256, 256, 2, 0.01
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=92)
    for px in (1, 8):
        with _env(MLP_PX=px):
            a = _train_gpu(mlp, d, B, lr, E, perm=d.perm)
        with _env(MLP_PX=px, MLP_FORCE_COHERENT=1):
            b = _train_gpu(mlp, d, B, lr, E, perm=d.perm)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


@pytest.mark.parametrize("strategy", ["tile", "optimized", "baseline"])
@pytest.mark.parametrize("h,B", [(256, 256), (1024, 1024), (32, 100)])
def test_host_loop_strategy_matches_oracle(mlp, strategy, h, B):
    _check_grad(mlp, h, B, n=5000, seed=3, strategy=strategy)
    n, E, lr = 1500, 2, 0.01
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=93 + h)
    g1, g2, gsl, gel = _train_gpu(mlp, d, B, lr, E, perm=d.perm, strategy=strategy)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, lr, E, perm=d.perm)
    check("W1 - W1_0", g1 - d.W1, ref["W1"] - d.W1.astype(np.float64), 1e-3)
    check("W2 - W2_0", g2 - d.W2, ref["W2"] - d.W2.astype(np.float64), 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-3 * ref["epoch_loss"])


@pytest.mark.parametrize("strategy", ["optimized", "baseline"])
@pytest.mark.parametrize("B", [1, 7, 64, 160, 1000])
def test_paper_strategy_small_batches(mlp, strategy, B):
    for h in (32, 256, 1024):
        _check_grad(mlp, h, B, seed=B, strategy=strategy)


@pytest.mark.parametrize("strategy", ["optimized", "baseline"])
def test_paper_strategy_worked_step_exact(mlp, strategy):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_two_sample.json")))
    X, W1, W2 = _embed(np.array(g["X"], np.float32), np.array(g["W1"]), np.array(g["W2"]), 256)
    Y = np.array(g["Y"], np.float32)
    ctx, w1, w2 = _ctx(mlp, W1, W2, 2, strategy)
    dW1, dW2, loss = mlp.mlp_backward(ctx, _to(X), _to(Y))
    exp1 = np.zeros((32, 256)); exp1[:2, :2] = g["dW1"]
    exp2 = np.zeros(256); exp2[:2] = g["dW2"]
    assert np.array_equal(dW1.cpu().numpy(), exp1) and np.array_equal(dW2.cpu().numpy(), exp2)
    assert float(loss.cpu()[0]) == g["loss"]


def test_paper_strategies_agree_bitwise(mlp):
    """The two strategies of the paper form every output with the same products
    in the same k order (only where operands live differs), so a training run
    gives bitwise equal weights and losses under both."""
    n, h, B, E, lr = 2560, 256, 256, 2, 0.002
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=94)
    a = _train_gpu(mlp, d, B, lr, E, perm=d.perm, strategy="optimized")
    b = _train_gpu(mlp, d, B, lr, E, perm=d.perm, strategy="baseline")
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_strategy_workspace_checks(mlp):
    d = datagen.make_data(64, 256, seed=4, with_perm=False)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, 256)
    need = mlp.mlp_strategy_workspace_bytes(32, 256, 256, mlp.STRATEGY_OPTIMIZED)
    assert need > 0 and need % 256 == 0
    assert mlp.mlp_strategy_workspace_bytes(32, 256, 256, mlp.STRATEGY_FUSED) == 0
    small = torch.empty(need - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):              # the binding's own size check
        mlp.mlp_set_strategy(ctx, "optimized", small)
    lib = mlp.load()                             # the library's check, past the binding
    assert lib.mlp_set_strategy(ctx.handle, mlp.STRATEGY_OPTIMIZED, small.data_ptr(),
                                small.numel()) == -3
    assert lib.mlp_set_strategy(ctx.handle, mlp.STRATEGY_OPTIMIZED, None, 0) == -3
    with pytest.raises(mlp.MLPError):
        mlp.mlp_set_strategy(ctx, 7)
    wg, launches = mlp.mlp_launch_info(ctx, 2560, 256, 100)
    assert launches == 1                        # still the fused strategy
    mlp.mlp_set_strategy(ctx, "baseline")
    wg, launches = mlp.mlp_launch_info(ctx, 2560, 256, 100)
    assert launches == 11 * 10 * 100 + 1


def test_launch_info_single_launch(mlp):
    d = datagen.make_data(64, 256, seed=4, with_perm=False)
    ctx, _, _ = _ctx(mlp, d.W1, d.W2, 4096)
    wg, launches = mlp.mlp_launch_info(ctx, 10_000_000, 4096, 3)
    assert launches == 1 and wg == 256
    mlp.mlp_set_strategy(ctx, "tile")
    wg, launches = mlp.mlp_launch_info(ctx, 10_000, 4096, 3)
    assert launches == 2 * 3 * 3 + 1


def test_batch_beyond_the_fused_shapes_runs_the_tile_path(mlp):
    """A batch of 6,000 rows at h = 256 is more than any fused trainer shape
    holds (4,096 rows), so mlp_train_epochs under the default strategy runs the
    tile path (two launches a step): one shuffled epoch of 20,000 rows (four
    steps, the last batch 2,000 rows) against the oracle at the main bars."""
    n, h, B, lr = 20000, 256, 6000, 0.002
    d = datagen.make_data(n, h, epochs=1, shuffle=True, seed=66)
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, B)
    wg, launches = mlp.mlp_launch_info(ctx, n, B, 1)
    assert launches == 2 * 4 + 1, launches
    g1, g2, gsl, gel = _train_gpu(mlp, d, B, lr, 1, perm=d.perm)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, lr, 1, perm=d.perm)
    assert ref["steps"] == 4 and len(gsl) == 4
    W10, W20 = d.W1.astype(np.float64), d.W2.astype(np.float64)
    check("W1 - W1_0", g1 - W10, ref["W1"] - W10, 1e-3)
    check("W2 - W2_0", g2 - W20, ref["W2"] - W20, 1e-3)
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * np.abs(ref["step_loss"]))
    assert abs(gel[0] - ref["epoch_loss"][0]) <= 1e-3 * ref["epoch_loss"][0]


@pytest.mark.parametrize("h,B", [(256, 4096), (1024, 1024), (32, 256)])
def test_zero_learning_rate(mlp, h, B):
    """lr = 0 (eq. 19 with a zero step): every step leaves W1 and W2 bitwise as
    they were, and each step's reported loss is the batch MSE at the initial
    weights (eq. 14), which the oracle's run with lr = 0 gives step by step."""
    n = 3 * B + B // 3
    d = datagen.make_data(n, h, epochs=1, shuffle=True, seed=h + B)
    g1, g2, gsl, gel = _train_gpu(mlp, d, B, 0.0, 1, perm=d.perm)
    assert np.array_equal(g1, d.W1) and np.array_equal(g2, d.W2)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, 0.0, 1, perm=d.perm)
    assert ref["steps"] == 4 and len(gsl) == 4
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-5 * ref["step_loss"])
    assert abs(gel[0] - ref["epoch_loss"][0]) <= 1e-5 * ref["epoch_loss"][0]


def test_workspace_reused_by_a_new_context(mlp):
    """A workspace that held another context's exchange words must not leak them
    into a new context (regression: stale step tags matched the new call's tags)."""
    d = datagen.make_data(5000, 256, epochs=1, shuffle=True, seed=61)
    need = mlp.mlp_workspace_bytes(32, 256, 4096)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    X, Y = _to(d.X), _to(d.Y)
    for trial in range(3):
        w1 = _to(d.W1)
        w2 = _to(d.W2)
        ctx = mlp.mlp_init(w1, w2, 4096, workspace=ws)
        if trial == 0:
            mlp.mlp_train_epochs(ctx, X, Y, 1000, 0.01, 1, perm=_to(d.perm))
        idx = np.arange(4096, dtype=np.int32)
        w1.copy_(_to(d.W1))
        w2.copy_(_to(d.W2))
        dW1, dW2, _ = mlp.mlp_backward(ctx, X, Y, _to(idx))
        torch.cuda.synchronize()
        mlp.mlp_check_errors(ctx)
        r1, r2, _, z, zabs = oracle.grad(d.X, d.Y, d.W1, d.W2, idx=idx, want_z=True)
        yp = oracle.forward(d.X, d.W1, d.W2, idx=idx)
        g1 = dW1.cpu().numpy()
        r1a, _, _ = align_kinks(g1, r1, d.X, d.Y, d.W1.astype(np.float64),
                                d.W2.astype(np.float64), idx, z, zabs, yp)
        assert rel(g1, r1a) <= 1e-4 and rel(dW2.cpu().numpy(), r2) <= 1e-4
        del ctx


@pytest.mark.parametrize("strategy", [None, "tile", "optimized", "baseline"])
def test_divergence_is_flagged(mlp, strategy):
    """A learning rate of 1e30 sends the weights to ~1e30 after the first step,
    so the next batch loss overflows: mlp_check_errors reports MLP_ERR_NONFINITE
    (and clears it). A finite run afterwards raises nothing."""
    d = datagen.make_data(2048, 256, epochs=1, shuffle=True, seed=71)
    print("strategy", strategy, flush=True)
    ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, 256, strategy)
    X, Y, P = _to(d.X), _to(d.Y), _to(d.perm)
    mlp.mlp_train_epochs(ctx, X, Y, 256, 1e30, 1, perm=P)
    with pytest.raises(mlp.MLPError) as e:
        mlp.mlp_check_errors(ctx)
    assert e.value.status == -5
    mlp.mlp_check_errors(ctx)                       # the check cleared the flag
    w1.copy_(_to(d.W1))
    w2.copy_(_to(d.W2))
    sl = torch.zeros(8, dtype=torch.float32, device="cuda")
    mlp.mlp_train_epochs(ctx, X, Y, 256, 0.002, 1, perm=P, step_loss=sl)
    mlp.mlp_check_errors(ctx)
    assert np.all(np.isfinite(sl.cpu().numpy()))


def test_tag_range_wrap_clears_and_restarts(mlp):
    """A context whose step tags start 20 below 2^32: the first 10-step call fits,
    the second would wrap, so the library clears the exchange words and restarts
    the tags at 1. Both calls give bitwise what a context with fresh tags gives."""
    n, h, B, lr = 4096, 256, 256, 0.01
    d = datagen.make_data(n, h, epochs=1, shuffle=True, seed=81)
    X, Y, P = _to(d.X), _to(d.Y), _to(d.perm)
    runs = []
    for base in (None, str(2 ** 32 - 20)):
        with _env(MLP_TAG_BASE=base):
            ctx, w1, w2 = _ctx(mlp, d.W1, d.W2, B)
        out = []
        for call in range(2):
            sl = torch.zeros(10, dtype=torch.float32, device="cuda")
            mlp.mlp_train_epochs(ctx, X, Y, B, lr, 1, perm=P, max_steps=10, step_loss=sl)
            torch.cuda.synchronize()
            mlp.mlp_check_errors(ctx)
            out.append((w1.cpu().numpy(), w2.cpu().numpy(), sl.cpu().numpy()))
        runs.append(out)
    for a, b in zip(runs[0], runs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
