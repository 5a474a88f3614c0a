"""Pins for the fp64 oracle, checked against facts fixed outside the oracle.

Each test ties the oracle to something it cannot agree with by construction:
finite differences of its own loss, the closed form of an all-active (linear)
net, hand-worked exact values, the strict ReLU'(0) = 0 convention, torch
float64 autograd, and invariants of the 2/n batch scaling. Paper equations:
Sec. III eqs. (11)-(19) (same as Sec. II.A eqs. (1)-(9)).
"""
import json
import os

import numpy as np
import pytest

import datagen
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rng(seed):
    return np.random.default_rng(seed)


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# --- hand-worked step (eqs. 11-19) -------------------------------------------

def test_worked_two_sample_step():
    g = _load("worked_two_sample.json")
    X = np.array(g["X"], np.float32)
    Y = np.array(g["Y"], np.float32)
    W1 = np.array(g["W1"])
    W2 = np.array(g["W2"])
    yp = oracle.forward(X, W1, W2)
    assert np.array_equal(yp, g["Ypred"])
    dW1, dW2, L, z, _ = oracle.grad(X, Y, W1, W2, want_z=True)
    assert np.array_equal(z, g["Z1"])
    assert L == g["loss"]
    assert np.array_equal(dW2, g["dW2"])
    assert np.array_equal(dW1, g["dW1"])
    out = oracle.train(X, Y, W1, W2, batch=2, lr=g["lr"], epochs=1)
    assert out["steps"] == 1
    np.testing.assert_allclose(out["W1"], g["W1_next"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(out["W2"], g["W2_next"], rtol=0, atol=1e-15)
    assert out["step_loss"][0] == g["loss"]
    assert out["epoch_loss"][0] == g["loss"]


def test_relu_prime_at_zero_is_zero():
    g = _load("relu_zero.json")
    X = np.array(g["X"], np.float32)
    Y = np.array(g["Y"], np.float32)
    dW1, dW2, L, z, _ = oracle.grad(X, Y, np.array(g["W1"]), np.array(g["W2"]), want_z=True)
    assert np.array_equal(z, g["Z1"])
    assert L == g["loss"]
    assert np.array_equal(dW1, g["dW1"]) and np.array_equal(dW2, g["dW2"])
    assert not np.array_equal(dW1, g["dW1_if_relu_prime_0_were_1"])


# --- finite differences on a 4-8-1 net ---------------------------------------

def _fd_case(seed, d=4, h=8, nb=5):
    rng = _rng(seed)
    while True:
        X = rng.standard_normal((nb, d)).astype(np.float32)
        Y = rng.standard_normal(nb).astype(np.float32)
        W1 = rng.standard_normal((d, h))
        W2 = rng.standard_normal(h)
        z = X.astype(np.float64) @ W1
        if np.min(np.abs(z)) > 1e-3:
            return X, Y, W1, W2


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_finite_differences_4_8_1(seed):
    X, Y, W1, W2 = _fd_case(seed)
    dW1, dW2, _ = oracle.grad(X, Y, W1, W2)
    eps = 1e-6

    def loss(a, b):
        return oracle.grad(X, Y, a, b)[2]

    fd1 = np.zeros_like(W1)
    for k in range(W1.shape[0]):
        for j in range(W1.shape[1]):
            p = W1.copy(); p[k, j] += eps
            m = W1.copy(); m[k, j] -= eps
            fd1[k, j] = (loss(p, W2) - loss(m, W2)) / (2 * eps)
    fd2 = np.zeros_like(W2)
    for j in range(W2.shape[0]):
        p = W2.copy(); p[j] += eps
        m = W2.copy(); m[j] -= eps
        fd2[j] = (loss(W1, p) - loss(W1, m)) / (2 * eps)
    assert _rel(dW1, fd1) < 1e-7
    assert _rel(dW2, fd2) < 1e-7


# --- closed form of an all-active net -----------------------------------------

def test_all_active_closed_form():
    rng = _rng(7)
    d, h, nb = 32, 256, 300
    X = np.abs(rng.standard_normal((nb, d))).astype(np.float32)
    Y = rng.standard_normal(nb).astype(np.float32)
    W1 = np.abs(rng.standard_normal((d, h))) * np.sqrt(2.0 / d) + 1e-3
    W2 = rng.standard_normal(h) * np.sqrt(2.0 / h)
    Xd = X.astype(np.float64)
    # With every pre-activation positive the net is linear: Ypred = X W1 W2.
    A = Xd @ W1
    assert A.min() > 0
    yp = A @ W2
    g = (2.0 / nb) * (yp - Y.astype(np.float64))
    dW2_cf = A.T @ g
    dW1_cf = Xd.T @ np.outer(g, W2)
    L_cf = np.mean((yp - Y) ** 2)
    dW1, dW2, L = oracle.grad(X, Y, W1, W2)
    assert _rel(dW1, dW1_cf) < 1e-12
    assert _rel(dW2, dW2_cf) < 1e-12
    assert abs(L - L_cf) <= 1e-12 * L_cf
    assert _rel(oracle.forward(X, W1, W2), yp) < 1e-13


# --- torch float64 autograd at the real shapes --------------------------------

def _torch_grad(X, Y, W1, W2):
    torch = pytest.importorskip("torch")
    x = torch.tensor(X, dtype=torch.float64)
    y = torch.tensor(Y, dtype=torch.float64)
    w1 = torch.tensor(W1, dtype=torch.float64, requires_grad=True)
    w2 = torch.tensor(W2, dtype=torch.float64, requires_grad=True)
    yp = torch.relu(x @ w1) @ w2
    L = torch.mean((yp - y) ** 2)
    L.backward()
    return w1.grad.numpy(), w2.grad.numpy(), float(L.detach())


@pytest.mark.parametrize("h,nb", [(256, 4096), (1024, 512), (32, 257)])
def test_torch_autograd_real_shapes(h, nb):
    data = datagen.make_data(nb, h, epochs=1, shuffle=False, seed=11 + h)
    W1 = data.W1.astype(np.float64)
    W2 = data.W2.astype(np.float64)
    dW1, dW2, L = oracle.grad(data.X, data.Y, W1, W2)
    t1, t2, tL = _torch_grad(data.X, data.Y, W1, W2)
    assert _rel(dW1, t1) < 1e-12
    assert _rel(dW2, t2) < 1e-12
    assert abs(L - tL) <= 1e-12 * tL


def test_torch_sgd_loop_with_shuffle_and_tail():
    """The epoch/batch/tail/update structure against an independent torch loop."""
    torch = pytest.importorskip("torch")
    n, h, B, E, lr = 1000, 64, 64, 3, 0.05        # tail batch of 40 rows
    data = datagen.make_data(n, h, epochs=E, shuffle=True, seed=5)
    out = oracle.train(data.X, data.Y, data.W1, data.W2, B, lr, E, perm=data.perm)
    x = torch.tensor(data.X, dtype=torch.float64)
    y = torch.tensor(data.Y, dtype=torch.float64)
    w1 = torch.tensor(data.W1, dtype=torch.float64)
    w2 = torch.tensor(data.W2, dtype=torch.float64)
    losses, epoch_losses = [], []
    for e in range(E):
        order = torch.tensor(data.perm[e], dtype=torch.long)
        sse = 0.0
        for s in range(0, n, B):
            rows = order[s:s + B]
            a = w1.clone().requires_grad_(True)
            b = w2.clone().requires_grad_(True)
            L = torch.mean((torch.relu(x[rows] @ a) @ b - y[rows]) ** 2)
            L.backward()
            with torch.no_grad():
                w1 = w1 - lr * a.grad
                w2 = w2 - lr * b.grad
            losses.append(float(L.detach()))
            sse += float(L.detach()) * len(rows)
        epoch_losses.append(sse / n)
    assert out["steps"] == len(losses) == E * 16
    assert _rel(out["W1"], w1.numpy()) < 1e-12
    assert _rel(out["W2"], w2.numpy()) < 1e-12
    np.testing.assert_allclose(out["step_loss"], losses, rtol=1e-12)
    np.testing.assert_allclose(out["epoch_loss"], epoch_losses, rtol=1e-12)


def test_max_steps_stops_exactly():
    data = datagen.make_data(300, 32, epochs=2, shuffle=True, seed=3)
    full = oracle.train(data.X, data.Y, data.W1, data.W2, 64, 0.01, 2, perm=data.perm)
    part = oracle.train(data.X, data.Y, data.W1, data.W2, 64, 0.01, 2, perm=data.perm,
                        max_steps=7)
    assert full["steps"] == 10 and part["steps"] == 7
    np.testing.assert_array_equal(part["step_loss"], full["step_loss"][:7])


# --- invariants of the batch scaling -------------------------------------------

def test_row_duplication_leaves_gradient_unchanged():
    """n in eqs. (14)-(15) is the batch row count: duplicating every row is a no-op."""
    data = datagen.make_data(200, 64, seed=21, with_perm=False)
    W1, W2 = data.W1.astype(np.float64), data.W2.astype(np.float64)
    idx = np.arange(200, dtype=np.int32)
    a = oracle.grad(data.X, data.Y, W1, W2, idx=idx)
    b = oracle.grad(data.X, data.Y, W1, W2, idx=np.concatenate([idx, idx]))
    assert _rel(b[0], a[0]) < 1e-13 and _rel(b[1], a[1]) < 1e-13
    assert abs(a[2] - b[2]) < 1e-13 * a[2]


def test_batch_union_is_row_weighted_mean():
    data = datagen.make_data(500, 128, seed=22, with_perm=False)
    W1, W2 = data.W1.astype(np.float64), data.W2.astype(np.float64)
    i1 = np.arange(0, 137, dtype=np.int32)
    i2 = np.arange(137, 500, dtype=np.int32)
    g1 = oracle.grad(data.X, data.Y, W1, W2, idx=i1)
    g2 = oracle.grad(data.X, data.Y, W1, W2, idx=i2)
    gu = oracle.grad(data.X, data.Y, W1, W2, idx=np.concatenate([i1, i2]))
    for t in range(2):
        assert _rel(gu[t], (137 * g1[t] + 363 * g2[t]) / 500) < 1e-13
    assert abs(gu[2] - (137 * g1[2] + 363 * g2[2]) / 500) < 1e-13 * gu[2]


def test_zero_output_weights_give_zero_dW1():
    data = datagen.make_data(64, 256, seed=23, with_perm=False)
    W2 = np.zeros(256)
    dW1, dW2, L = oracle.grad(data.X, data.Y, data.W1.astype(np.float64), W2)
    assert np.all(dW1 == 0.0)
    assert np.any(dW2 != 0.0)
    assert abs(L - np.mean(data.Y.astype(np.float64) ** 2)) < 1e-14


def test_all_inactive_gives_zero_everything():
    rng = _rng(24)
    X = np.abs(rng.standard_normal((50, 32))).astype(np.float32)
    Y = rng.standard_normal(50).astype(np.float32)
    W1 = -np.abs(rng.standard_normal((32, 256)))
    W2 = rng.standard_normal(256)
    assert np.all(oracle.forward(X, W1, W2) == 0.0)
    dW1, dW2, _ = oracle.grad(X, Y, W1, W2)
    assert np.all(dW1 == 0.0) and np.all(dW2 == 0.0)


def test_small_full_batch_step_decreases_loss():
    data = datagen.make_data(512, 256, seed=25, with_perm=False)
    W1, W2 = data.W1.astype(np.float64), data.W2.astype(np.float64)
    dW1, dW2, L0 = oracle.grad(data.X, data.Y, W1, W2)
    _, _, L1 = oracle.grad(data.X, data.Y, W1 - 1e-3 * dW1, W2 - 1e-3 * dW2)
    assert L1 < L0


def test_parameter_count_eq10():
    data = datagen.make_data(4, 256, seed=0, with_perm=False)
    assert data.W1.size + data.W2.size == 8448


def test_bad_arguments_are_rejected():
    data = datagen.make_data(8, 32, seed=0, with_perm=False)
    W1, W2 = data.W1.astype(np.float64), data.W2.astype(np.float64)
    with pytest.raises(ValueError):
        oracle.grad(data.X, data.Y, W1, W2, idx=np.array([0, 8], np.int32))
    with pytest.raises(ValueError):
        oracle.grad(data.X, data.Y, W1, W2, idx=np.array([-1], np.int32))
