"""fp32 on device: the split products are at least as accurate as plain fp32.

The trainer, the forward pass and the deep path's 64 x 64 GEMM tiles form their
fp32 products on the bf16 matrix cores: every fp32 operand is split exactly
into three bf16 parts, the six part products with i + j <= 2 (each exact in
fp32) are accumulated in fp32, and only the three smallest part products (at
most 2.01 u |x y| together, u = 2^-24) are dropped. Data, accumulation and
results are fp32; this is not a reduced-precision substitute for fp32.

These tests put that to a measurement on the evaluation workloads' data: the
device's results and those of a plain fp32 computation of the same equations
(numpy float32, BLAS sgemm; eqs. 11-18, and the same for L hidden layers) are
both compared with the fp64 oracle, and the device's error must not exceed the
plain fp32 one by more than half (measured: 0.13-0.70 of it). Gradients of
the one-layer net are kink-aligned on both sides (tests/parity.py); the deep
case uses kink-free rows (tests/test_gpu_deep.py).
"""
import numpy as np
import pytest
import torch

import datagen
import oracle
from tests.parity import align_kinks, rel, relmax
from tests.test_gpu_deep import _gauss_net, _kink_free

pytestmark = pytest.mark.gpu

RATIO = 1.5   # device error / plain fp32 error, normwise and max elementwise


@pytest.fixture(scope="module")
def mlp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_30497_amd import mlp as m
    m.load(require_built=True)
    return m


def _to(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _f32_step(X, Y, W1, W2):
    """Eqs. 11-18 in plain fp32 (numpy float32): Ypred, dW1, dW2."""
    f = np.float32
    X, Y, W1, W2 = X.astype(f), Y.astype(f), W1.astype(f), W2.astype(f)
    Z = X @ W1
    H = np.maximum(Z, f(0))
    yp = H @ W2
    g = (f(2.0 / X.shape[0]) * (yp - Y)).astype(f)
    dW2 = H.T @ g
    dZ = (np.outer(g, W2) * (Z > 0)).astype(f)
    return yp, X.T @ dZ, dW2


def _compare(name, dev, f32, ref, ref_f32=None):
    """Errors of the device's and the plain fp32 result against the fp64
    reference (ref_f32: the reference aligned to the fp32 result's own mask
    choices, where that differs)."""
    rf = ref if ref_f32 is None else ref_f32
    ed, md = rel(dev, ref), relmax(dev, ref)
    ef, mf = rel(f32, rf), relmax(f32, rf)
    print("%-22s device rel %.3e relmax %.3e | plain fp32 rel %.3e relmax %.3e | ratio %.2f %.2f"
          % (name, ed, md, ef, mf, ed / ef, md / mf), flush=True)
    assert ed <= RATIO * ef, (name, "normwise", ed, ef)
    assert md <= RATIO * mf, (name, "max elementwise", md, mf)


@pytest.mark.parametrize("k", [4, 3])   # 32-256-1 at batch 4096; 32-1024-1 at batch 1024
def test_trainer_and_forward_at_fp32_level(mlp, k):
    w = datagen.WORKLOADS[k]
    n = 200_000
    d = datagen.make_data(n, w.hidden, seed=w.seed, with_perm=False)
    B = w.batch
    idx = np.random.default_rng(7).integers(0, n, size=B).astype(np.int32)
    ctx = mlp.mlp_init(_to(d.W1), _to(d.W2), B)
    dW1, dW2, _ = mlp.mlp_backward(ctx, _to(d.X), _to(d.Y), _to(idx), B=B)
    yp = mlp.mlp_forward(ctx, _to(d.X), _to(idx)).cpu().numpy()
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    g1, g2 = dW1.cpu().numpy(), dW2.cpu().numpy()
    W1, W2 = d.W1.astype(np.float64), d.W2.astype(np.float64)
    r1, r2, _, z, zabs = oracle.grad(d.X, d.Y, W1, W2, idx=idx, nb=B, want_z=True)
    ry = oracle.forward(d.X, W1, W2, idx=idx, nb=B)
    fy, f1, f2 = _f32_step(d.X[idx], d.Y[idx], d.W1, d.W2)
    r1g, _, _ = align_kinks(g1, r1, d.X, d.Y, W1, W2, idx, z, zabs, ry)
    r1f, _, _ = align_kinks(f1, r1, d.X, d.Y, W1, W2, idx, z, zabs, ry)
    _compare("Ypred (h=%d)" % w.hidden, yp, fy, ry)
    _compare("dW2 (h=%d)" % w.hidden, g2, f2, r2)
    _compare("dW1 (h=%d)" % w.hidden, g1, f1, r1g, r1f)


def _f32_deep(X, Y, P, h, L):
    """The L-layer step in plain fp32: Ypred and the flat gradient."""
    f = np.float32
    Ws, wo = oracle.deep_split(np.asarray(P, np.float64), 32, h, L)
    Ws = [W.astype(f) for W in Ws]
    wo = wo.astype(f)
    Hs = [X.astype(f)]
    for W in Ws:
        Hs.append(np.maximum(Hs[-1] @ W, f(0)))
    yp = Hs[-1] @ wo
    g = (f(2.0 / X.shape[0]) * (yp - Y.astype(f))).astype(f)
    dwo = Hs[-1].T @ g
    G = (np.outer(g, wo) * (Hs[-1] > 0)).astype(f)
    dWs = [None] * L
    for l in range(L, 0, -1):
        dWs[l - 1] = Hs[l - 1].T @ G
        if l > 1:
            G = ((G @ Ws[l - 1].T) * (Hs[l - 1] > 0)).astype(f)
    return yp, np.concatenate([dW.ravel() for dW in dWs] + [dwo])


def test_deep_wide_tiles_at_fp32_level(mlp):
    """32-1024x2-1 at a batch of 2100 kink-free rows: every product that runs
    64 x 64 tiles (the forward, the W_2 gradient paired with the
    back-propagation) is formed from split parts."""
    h, L, B = 1024, 2, 2100
    rng = np.random.default_rng(4096)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    rows = _kink_free(d.X, P, h, L, rng.integers(0, 5000, size=8 * B).astype(np.int32))[:B]
    assert len(rows) == B
    p = _to(P)
    ctx = mlp.mlp_deep_init(p, h, L, B)
    dP, _ = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(rows))
    yp = mlp.mlp_deep_forward(ctx, _to(d.X), _to(rows)).cpu().numpy()
    torch.cuda.synchronize()
    mlp.mlp_deep_check_errors(ctx)
    ref, _, _ = oracle.deep_grad(d.X, d.Y, P, 32, h, L, idx=rows)
    ry = oracle.deep_forward(d.X, P, 32, h, L, idx=rows)
    fy, fg = _f32_deep(d.X[rows], d.Y[rows], P, h, L)
    _compare("deep Ypred (h=1024)", yp, fy, ry)
    _compare("deep gradient (h=1024)", dP.cpu().numpy(), fg, ref)
