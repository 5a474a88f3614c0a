"""Pins of the L-hidden-layer oracle (oracle/oracle_deep.c) against facts that do
not come from the oracle itself:

- at L = 1 it is the paper's network, so it must agree with oracle.c (written
  separately and pinned by tests/test_oracle_pins.py) on gradients, losses and
  whole training runs;
- central finite differences of the loss on small deep nets;
- the closed form of an all-active net, which is linear (every ReLU passes its
  input): Ypred = X W_1 ... W_L w_o, and each gradient is an outer product of
  matrix-product chains computed with numpy;
- torch float64 autograd on the same network;
- ReLU'(0) = 0 through two layers (a hand-worked case).
"""
import numpy as np
import pytest

import oracle


def _rand_net(rng, d, h, L, scale=1.0):
    P = []
    for l in range(L):
        K = d if l == 0 else h
        P.append(rng.standard_normal(K * h) * np.sqrt(2.0 / K) * scale)
    P.append(rng.standard_normal(h) * np.sqrt(2.0 / h) * scale)
    return np.concatenate(P)


def _data(rng, n, d):
    X = rng.standard_normal((n, d)).astype(np.float32)
    Y = rng.standard_normal(n).astype(np.float32)
    return X, Y


def test_param_count():
    assert oracle.deep_param_count(32, 256, 1) == 32 * 256 + 256 == 8448   # eq. 10
    assert oracle.deep_param_count(32, 256, 3) == 32 * 256 + 2 * 256 * 256 + 256


@pytest.mark.parametrize("h", [8, 64, 256])
def test_one_layer_matches_the_shallow_oracle(h):
    rng = np.random.default_rng(h)
    d, n = 32, 300
    X, Y = _data(rng, n, d)
    P = _rand_net(rng, d, h, 1)
    W1, W2 = P[:d * h].reshape(d, h), P[d * h:]
    idx = rng.integers(0, n, size=77).astype(np.int32)
    dP, loss, _ = oracle.deep_grad(X, Y, P, d, h, 1, idx=idx)
    g1, g2, l1 = oracle.grad(X, Y, W1, W2, idx=idx)
    np.testing.assert_allclose(dP[:d * h].reshape(d, h), g1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dP[d * h:], g2, rtol=1e-12, atol=1e-15)
    assert abs(loss - l1) <= 1e-13 * abs(l1)
    np.testing.assert_allclose(oracle.deep_forward(X, P, d, h, 1, idx=idx),
                               oracle.forward(X, W1, W2, idx=idx), rtol=1e-13, atol=1e-15)
    perm = np.stack([rng.permutation(n) for _ in range(2)]).astype(np.int32)
    a = oracle.deep_train(X, Y, P, d, h, 1, 64, 0.01, 2, perm=perm)     # tail of 44 rows
    b = oracle.train(X, Y, W1, W2, 64, 0.01, 2, perm=perm)
    assert a["steps"] == b["steps"] == 10
    np.testing.assert_allclose(a["P"][:d * h].reshape(d, h), b["W1"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a["P"][d * h:], b["W2"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a["step_loss"], b["step_loss"], rtol=1e-12)
    np.testing.assert_allclose(a["epoch_loss"], b["epoch_loss"], rtol=1e-12)


def _loss(X, Y, P, d, h, L, idx):
    return float(np.mean((oracle.deep_forward(X, P, d, h, L, idx=idx)
                          - Y[idx].astype(np.float64)) ** 2))


@pytest.mark.parametrize("d,h,L,seed", [(4, 6, 2, 0), (4, 6, 3, 1), (5, 4, 4, 2)])
def test_finite_differences(d, h, L, seed):
    rng = np.random.default_rng(100 + seed)
    X, Y = _data(rng, 9, d)
    P = _rand_net(rng, d, h, L)
    idx = np.array([0, 3, 3, 8, 5, 1], np.int32)
    dP, loss, margin = oracle.deep_grad(X, Y, P, d, h, L, idx=idx)
    assert margin > 1e-4, "a pre-activation sits on the ReLU kink; pick another seed"
    assert abs(loss - _loss(X, Y, P, d, h, L, idx)) <= 1e-13 * loss
    eps = 1e-6
    fd = np.empty_like(P)
    for i in range(P.size):
        Pp, Pm = P.copy(), P.copy()
        Pp[i] += eps
        Pm[i] -= eps
        fd[i] = (_loss(X, Y, Pp, d, h, L, idx) - _loss(X, Y, Pm, d, h, L, idx)) / (2 * eps)
    np.testing.assert_allclose(dP, fd, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("L", [2, 3, 4])
def test_all_active_net_is_linear(L):
    """Positive inputs and weights: every pre-activation is positive, so H_l =
    X W_1 ... W_l and the gradients have closed forms:
      dw_o = H_L^T g,  dW_l = (H_{l-1}^T g) (W_{l+1} ... W_L w_o)^T,
    with g = (2/n)(Ypred - Y)."""
    rng = np.random.default_rng(L)
    d, h, nb = 32, 16, 23
    X = np.abs(rng.standard_normal((nb, d))).astype(np.float32)
    Y = rng.standard_normal(nb).astype(np.float32)
    P = np.abs(_rand_net(rng, d, h, L, scale=0.3))
    Ws, wo = oracle.deep_split(P, d, h, L)
    dP, loss, margin = oracle.deep_grad(X, Y, P, d, h, L)
    assert margin == 1.0                               # no cancellation: all terms positive
    Hs = [X.astype(np.float64)]
    for W in Ws:
        Hs.append(Hs[-1] @ W)
    yp = Hs[-1] @ wo
    g = 2.0 / nb * (yp - Y.astype(np.float64))
    assert abs(loss - np.mean((yp - Y) ** 2)) <= 1e-12 * loss
    dWs, dwo = oracle.deep_split(dP, d, h, L)
    np.testing.assert_allclose(dwo, Hs[-1].T @ g, rtol=1e-11)
    for l in range(L):
        tail = wo.copy()
        for W in reversed(Ws[l + 1:]):
            tail = W @ tail
        np.testing.assert_allclose(dWs[l], np.outer(Hs[l].T @ g, tail), rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("h,L", [(64, 2), (64, 3), (256, 3)])
def test_torch_autograd(h, L):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(h + L)
    d, n = 32, 200
    X, Y = _data(rng, n, d)
    P = _rand_net(rng, d, h, L)
    idx = rng.integers(0, n, size=41).astype(np.int32)
    dP, loss, margin = oracle.deep_grad(X, Y, P, d, h, L, idx=idx)
    assert margin > 1e-9
    Pt = torch.tensor(P, dtype=torch.float64, requires_grad=True)
    Xt = torch.tensor(X[idx], dtype=torch.float64)
    Yt = torch.tensor(Y[idx], dtype=torch.float64)
    Ws, wo = [], None
    off = 0
    for l in range(L):
        K = d if l == 0 else h
        Ws.append(Pt[off:off + K * h].reshape(K, h))
        off += K * h
    wo = Pt[off:off + h]
    Hc = Xt
    for W in Ws:
        Hc = torch.relu(Hc @ W)
    lt = torch.mean((Hc @ wo - Yt) ** 2)
    lt.backward()
    assert abs(lt.item() - loss) <= 1e-12 * loss
    np.testing.assert_allclose(dP, Pt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_relu_prime_at_zero_through_two_layers():
    """2-2-2-1 net, x = [1, -1], y = 1: Z_1 = [0, -0.5] exactly, so H_1 = 0,
    Z_2 = 0 and Ypred = 0, r = -1. With ReLU'(0) = 0 every gradient is zero;
    with ReLU'(0) = 1, dW_1[:, 0] would be [-4, 4]."""
    X = np.array([[1.0, -1.0]], np.float32)
    Y = np.array([1.0], np.float32)
    W1 = np.array([[1.0, 0.5], [1.0, 1.0]])
    W2 = np.ones((2, 2))
    wo = np.ones(2)
    P = np.concatenate([W1.ravel(), W2.ravel(), wo])
    dP, loss, margin = oracle.deep_grad(X, Y, P, 2, 2, 2)
    assert loss == 1.0 and margin == 0.0
    assert np.all(dP == 0.0)
