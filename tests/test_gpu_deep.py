"""GPU parity of the L-hidden-layer path (mlp_deep_*) against the deep oracle.

Two kinds of inputs:
- dyadic: X, Y and every weight are small multiples of 1/4, 1/8 or 1/16, chosen
  so that every pre-activation is an integer multiple of its scale whose
  partial sums stay below 2^24 of that scale. Then fp32 computes every Z
  exactly, in any summation order: the forward must match the oracle bitwise and
  the ReLU masks cannot differ, so the gradients are held to 1e-5 (only the
  backward's sums round);
- Gaussian (the evaluation-workload recipe): the forward and the loss are
  continuous at the ReLU kink and are held to 1e-5. An fp32 pre-activation
  within rounding of zero may take either mask value (a correct result either
  way), so the gradient checks run on the rows of the batch whose every
  pre-activation is farther from zero than a rigorous bound on the device's
  rounding error (_kink_free: then the device's masks are the exact ones) and
  hold them to 1e-5, ten times inside the main path's per-step bar. The bound compounds with
  depth, so at eight layers no row qualifies and the whole batch is held to
  1e-3; the 1024-wide large-tile case also keeps its whole batch (its point is
  the tile shapes of 2100 rows) and the 1e-3 bar. At L = 1 the network is the paper's
  and the gradients meet 1e-4 after the kink alignment of tests/parity.py.
"""
import numpy as np
import pytest
import torch

import datagen
import oracle
from tests.parity import U32, align_kinks, rel

pytestmark = pytest.mark.gpu

D = 32


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


def _gauss_net(rng, h, L):
    parts = []
    for l in range(L):
        K = D if l == 0 else h
        parts.append(rng.standard_normal(K * h) * np.sqrt(2.0 / K))
    parts.append(rng.standard_normal(h) * np.sqrt(2.0 / h))
    return np.concatenate(parts).astype(np.float32)


def _kink_free(X, P, h, L, idx):
    """The rows of idx whose pre-activations all lie farther from zero than a
    bound on the device's error. Layer l computes Z = H_{l-1} W_l, a sum of K
    products, from an input each entry of which is within e_{l-1} of exact
    (e_0 = 0: X is exact). The device forms each product a b from three-part
    bf16 splits of a and b (a = a0 + a1 + a2 exactly, |a1| <= 2^-8 (1 + 2^-8)|a|,
    |a2| <= 2^-16 |a|): a0 b0 summed over k in fp32 (K terms, within
    (1 + 2^-8)^2 |a b| each: at most 1.016 K u sum |a b| of rounding), the five
    part products with i + j in {1, 2} in a second fp32 sum (5 K terms, below
    1.02 * 2^-7 |a b| per k together: at most 0.04 K u), one addition of the
    two (1.02 u) and the three dropped part products (at most 2.01 u |a b|).
    So the device's Z is within
    e_l = (1.1 K + 4) u sum_k (|H_k| + e_k) |W_kj| + sum_k e_k |W_kj| of exact
    (each term is also off by at most e_k |W_kj| through its input; ReLU is
    1-Lipschitz, so e_l also bounds the layer's output). Where |Z| > e_l the
    device's ReLU mask equals the exact one."""
    Ws, _ = oracle.deep_split(np.asarray(P, np.float64), D, h, L)
    Hp = np.asarray(X, np.float64)[idx]
    Ep = np.zeros_like(Hp)
    ok = np.ones(len(idx), bool)
    for W in Ws:
        K = W.shape[0]
        A = np.abs(W)
        Z = Hp @ W
        prop = Ep @ A
        E = (1.1 * K + 4) * U32 * (np.abs(Hp) @ A + prop) + prop
        ok &= np.all(np.abs(Z) > E, axis=1)
        Hp, Ep = np.maximum(Z, 0.0), E
    return np.ascontiguousarray(idx[ok])


def _dyadic(rng, n, h, L):
    """Integer numerators with scales 1/4 (X), 1/16 (weights), 1/8 (Y). The
    forward is run in exact integer arithmetic to check that, for every
    pre-activation and for Ypred, the sum of the terms' magnitudes (a bound on
    every partial sum, in units of the entry's scale) stays below 2^24."""
    Xi = rng.integers(-3, 4, size=(n, D)).astype(np.int64)
    Wi = [rng.integers(-3, 4, size=(D if l == 0 else h, h)).astype(np.int64) for l in range(L)]
    woi = rng.integers(-3, 4, size=h).astype(np.int64)
    Hi = Xi
    for W in Wi:
        assert (np.abs(Hi) @ np.abs(W)).max() < 2 ** 24
        Hi = np.maximum(Hi @ W, 0)
    assert (Hi @ np.abs(woi)).max() < 2 ** 24
    X = (Xi / 4.0).astype(np.float32)
    Y = (rng.integers(-8, 9, size=n) / 8.0).astype(np.float32)
    P = np.concatenate([W.ravel() / 16.0 for W in Wi] + [woi / 16.0]).astype(np.float32)
    return X, Y, P


def _ctx(mlp, P, h, L, max_batch):
    p = _to(P.astype(np.float32))
    return mlp.mlp_deep_init(p, h, L, max_batch), p


# --- forward -------------------------------------------------------------------

@pytest.mark.parametrize("h,L", [(64, 1), (64, 2), (64, 3), (128, 2), (192, 2)])
def test_forward_dyadic_is_exact(mlp, h, L):
    rng = np.random.default_rng(10 * h + L)
    X, Y, P = _dyadic(rng, 1000, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 256)             # 1000 rows: four chunks of max_batch
    got = mlp.mlp_deep_forward(ctx, _to(X)).cpu().numpy()
    ref = oracle.deep_forward(X, P, D, h, L)
    assert np.array_equal(got, ref.astype(np.float32))
    mlp.mlp_deep_check_errors(ctx)


def test_forward_dyadic_is_exact_wide_tiles(mlp):
    """h = 1024 at 2100 rows: the forward products run 64 x 64 tiles, the bf16x3
    flavour (three-part bf16 splits on the bf16 matrix cores); on dyadic inputs
    every part product and partial sum is exact, so the output must match the
    oracle bitwise, as in the fp32 flavour."""
    h, L = 1024, 2
    rng = np.random.default_rng(1024)
    X, Y, P = _dyadic(rng, 2100, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 2100)
    got = mlp.mlp_deep_forward(ctx, _to(X)).cpu().numpy()
    ref = oracle.deep_forward(X, P, D, h, L)
    assert np.array_equal(got, ref.astype(np.float32))
    mlp.mlp_deep_check_errors(ctx)


@pytest.mark.parametrize("h,L", [(64, 2), (256, 3), (1024, 2)])
def test_forward_gaussian(mlp, h, L):
    rng = np.random.default_rng(h + L)
    d = datagen.make_data(3001, 32, seed=5, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 512)
    idx = rng.integers(0, 3001, size=1777).astype(np.int32)
    got = mlp.mlp_deep_forward(ctx, _to(d.X), _to(idx)).cpu().numpy()
    assert rel(got, oracle.deep_forward(d.X, P, D, h, L, idx=idx)) < 1e-5
    mlp.mlp_deep_check_errors(ctx)


# --- gradients -----------------------------------------------------------------

@pytest.mark.parametrize("h,L", [(64, 1), (64, 2), (64, 3), (128, 3)])
@pytest.mark.parametrize("B", [1, 16, 64, 256])
def test_gradients_dyadic(mlp, h, L, B):
    rng = np.random.default_rng(1000 * L + 7 * h + B)
    X, Y, P = _dyadic(rng, 600, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 256)
    idx = rng.integers(0, 600, size=B).astype(np.int32)
    dP, loss = mlp.mlp_deep_backward(ctx, _to(X), _to(Y), _to(idx))
    torch.cuda.synchronize()
    mlp.mlp_deep_check_errors(ctx)
    ref, rL, _ = oracle.deep_grad(X, Y, P, D, h, L, idx=idx)
    assert rel(dP.cpu().numpy(), ref) <= 1e-5
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * max(rL, 1e-30)


@pytest.mark.parametrize("h,L", [(64, 2), (256, 2), (256, 3)])
@pytest.mark.parametrize("B", [7, 160, 1000])
def test_gradients_gaussian(mlp, h, L, B):
    """Loss of a random batch at 1e-5; gradients of a batch of B kink-free rows
    (drawn from up to 8 B random rows) at 1e-5, as in the dyadic cases (measured
    0.7-7e-7: with the masks settled only the fp32 sums round)."""
    rng = np.random.default_rng(h * L + B)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 1024)
    idx = rng.integers(0, 5000, size=B).astype(np.int32)
    _, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(idx))
    _, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=idx)
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL
    cand = rng.integers(0, 5000, size=8 * B).astype(np.int32)
    rows = _kink_free(d.X, P, h, L, cand)[:B]
    assert len(rows) == B, (len(rows), B)
    dP, _ = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(rows))
    ref, _, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=rows)
    e = rel(dP.cpu().numpy(), ref)
    print("kink-free batch of %d rows: gradient rel %.3e" % (B, e))
    assert e <= 1e-5
    mlp.mlp_deep_check_errors(ctx)


def test_gradients_gaussian_wide_tiles(mlp):
    """h = 1024 with a batch of 2100 kink-free rows: every product of the step
    that runs 64 x 64 tiles (the forward, the W_2 gradient paired with the
    back-propagation) takes the bf16x3 flavour; gradients and loss at 1e-5 as
    in the fp32-flavour cases (one oracle pass: 2100 rows at h = 1024 take the
    fp64 oracle about 16 s)."""
    h, L, B = 1024, 2, 2100
    rng = np.random.default_rng(4096)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, B)
    cand = rng.integers(0, 5000, size=8 * B).astype(np.int32)
    rows = _kink_free(d.X, P, h, L, cand)[:B]
    assert len(rows) == B, (len(rows), B)
    dP, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(rows))
    ref, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=rows)
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL
    e = rel(dP.cpu().numpy(), ref)
    print("kink-free batch of %d rows at h = 1024: gradient rel %.3e" % (B, e))
    assert e <= 1e-5
    mlp.mlp_deep_check_errors(ctx)


@pytest.mark.parametrize("h", [192, 320, 960])
def test_widths_off_the_power_of_two_grid(mlp, h):
    """Hidden widths with an odd number of 64-unit tiles (3, 5, 15): the GEMM
    grids' unit-tile counts, the output kernel's units per lane and the
    update kernel's segment ends all differ from the power-of-two nets. At a
    batch of 500 kink-free rows (ragged against every row tile): the forward at
    1e-5, gradients and loss at 1e-5, and two SGD steps against the oracle's."""
    L, B, lr = 2, 500, 0.002
    rng = np.random.default_rng(h)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, p = _ctx(mlp, P, h, L, B)
    cand = rng.integers(0, 5000, size=8 * B).astype(np.int32)
    rows = _kink_free(d.X, P, h, L, cand)[:B]
    assert len(rows) == B, (len(rows), B)
    got = mlp.mlp_deep_forward(ctx, _to(d.X), _to(rows)).cpu().numpy()
    assert rel(got, oracle.deep_forward(d.X, P, D, h, L, idx=rows)) < 1e-5
    dP, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(rows))
    ref, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=rows)
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL
    e = rel(dP.cpu().numpy(), ref)
    print("h = %d, kink-free batch of %d rows: gradient rel %.3e" % (h, B, e))
    assert e <= 1e-5
    # two steps over a 1000-row set in identity order (batches of 500)
    X2, Y2 = d.X[:1000], d.Y[:1000]
    gP, gsl, _ = _train(mlp, X2, Y2, P, h, L, B, lr, 1, max_steps=2)
    tr = oracle.deep_train(X2, Y2, P, D, h, L, B, lr, 1, max_steps=2)
    P0 = P.astype(np.float64)
    assert rel(gP - P0, tr["P"] - P0) <= 1e-3
    assert np.all(np.abs(gsl - tr["step_loss"]) <= 1e-4 * tr["step_loss"])
    mlp.mlp_deep_check_errors(ctx)


def test_large_batch_split_plans(mlp):
    """A batch of 20,000 kink-free rows at 32-256x2-1: the back-propagation runs
    64 x 64 tiles beside a weight gradient on 32 x 64 tiles (16 row chunks of
    1280 rows, the last one ragged) in one launch, dW_1 comes in 313 partials
    (one per 64-row tile), and the output layer in 209 chunks of 96 rows (its
    cap of 256 chunks reached), so the update kernel's loops run many batches
    and a tail. Gradient and loss at 1e-5."""
    h, L, B = 256, 2, 20000
    rng = np.random.default_rng(20000)
    d = datagen.make_data(60000, 32, seed=8, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, B)
    cand = rng.integers(0, 60000, size=2 * B).astype(np.int32)
    rows = _kink_free(d.X, P, h, L, cand)[:B]
    assert len(rows) == B, (len(rows), B)
    dP, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(rows))
    ref, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=rows)
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL
    e = rel(dP.cpu().numpy(), ref)
    print("kink-free batch of %d rows: gradient rel %.3e" % (B, e))
    assert e <= 1e-5
    mlp.mlp_deep_check_errors(ctx)


@pytest.mark.parametrize("h,L", [(64, 8), (128, 8)])
@pytest.mark.parametrize("B", [7, 160, 1000])
def test_gradients_gaussian_eight_layers(mlp, h, L, B):
    """Eight layers: the rounding bound of _kink_free compounds with depth
    (each layer multiplies it by about sum_k |W_kj|), so no row is provably
    kink-free; the whole batch is compared at 1e-3, the loss at 1e-5."""
    rng = np.random.default_rng(h * L + B)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, 1024)
    idx = rng.integers(0, 5000, size=B).astype(np.int32)
    dP, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(idx))
    ref, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=idx)
    assert rel(dP.cpu().numpy(), ref) <= 1e-3
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL


@pytest.mark.parametrize("B", [2100])
def test_large_tiles(mlp, B):
    """h = 1024 at a batch of 2100 rows: the forward and back-propagation
    products run 64 x 64 tiles (33 x 16 of them, the last one 52 rows deep),
    the launch shapes of the 1024-wide evaluation net (smaller batches run
    32 x 64 tiles); the W_2 gradient runs two row chunks of 64 x 64 tiles.
    Gradients and loss against the oracle as in the other Gaussian cases; the
    forward of all B rows on sampled rows."""
    h, L = 1024, 2
    rng = np.random.default_rng(21 + B)
    d = datagen.make_data(5000, 32, seed=6, with_perm=False)
    P = _gauss_net(rng, h, L)
    ctx, _ = _ctx(mlp, P, h, L, B)
    idx = rng.integers(0, 5000, size=B).astype(np.int32)
    dP, loss = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(idx))
    ref, rL, _ = oracle.deep_grad(d.X, d.Y, P, D, h, L, idx=idx)
    assert rel(dP.cpu().numpy(), ref) <= 1e-3
    assert abs(float(loss.cpu()[0]) - rL) <= 1e-5 * rL
    got = mlp.mlp_deep_forward(ctx, _to(d.X), _to(idx)).cpu().numpy()
    rows = np.arange(0, B, 7 if B < 3000 else 13)
    assert rel(got[rows], oracle.deep_forward(d.X, P, D, h, L, idx=idx[rows])) < 1e-5
    mlp.mlp_deep_check_errors(ctx)


@pytest.mark.parametrize("h", [64, 256])
def test_one_layer_meets_the_main_bar(mlp, h):
    """L = 1 is the paper's network: gradients within 1e-4 of the shallow oracle
    after the kink alignment used for the main path."""
    d = datagen.make_data(5000, h, seed=300 + h, with_perm=False)
    P = np.concatenate([d.W1.ravel(), d.W2]).astype(np.float32)
    ctx, _ = _ctx(mlp, P, h, 1, 4096)
    idx = np.random.default_rng(h).integers(0, 5000, size=4096).astype(np.int32)
    dP, _ = mlp.mlp_deep_backward(ctx, _to(d.X), _to(d.Y), _to(idx))
    g = dP.cpu().numpy()
    W1, W2 = d.W1.astype(np.float64), d.W2.astype(np.float64)
    r1, r2, _, z, zabs = oracle.grad(d.X, d.Y, W1, W2, idx=idx, want_z=True)
    yp = oracle.forward(d.X, W1, W2, idx=idx)
    g1 = g[:D * h].reshape(D, h)
    r1a, _, _ = align_kinks(g1, r1, d.X, d.Y, W1, W2, idx, z, zabs, yp)
    assert rel(g1, r1a) <= 1e-4
    assert rel(g[D * h:], r2) <= 1e-4


# --- training ------------------------------------------------------------------

def _train(mlp, X, Y, P, h, L, batch, lr, epochs, perm=None, max_steps=-1):
    ctx, p = _ctx(mlp, P, h, L, batch)
    n = X.shape[0]
    steps = -(-n // batch) * epochs if max_steps < 0 else max_steps
    el = torch.zeros(epochs, dtype=torch.float32, device="cuda")
    sl = torch.zeros(steps, dtype=torch.float32, device="cuda")
    mlp.mlp_deep_train_epochs(ctx, _to(X), _to(Y), batch, lr, epochs,
                              perm=None if perm is None else _to(perm), max_steps=max_steps,
                              epoch_loss=el, step_loss=sl)
    torch.cuda.synchronize()
    mlp.mlp_deep_check_errors(ctx)
    return p.cpu().numpy(), sl.cpu().numpy(), el.cpu().numpy()


@pytest.mark.parametrize("h,L", [(64, 2), (64, 3), (256, 2)])
def test_train_epochs_with_shuffle_and_tail(mlp, h, L):
    n, B, E, lr = 1000, 128, 2, 2.0 ** -7                 # tail of 104 rows each epoch
    rng = np.random.default_rng(h + 10 * L)
    X, Y, P = _dyadic(rng, n, h, L)
    perm = np.stack([rng.permutation(n) for _ in range(E)]).astype(np.int32)
    gP, gsl, gel = _train(mlp, X, Y, P, h, L, B, lr, E, perm=perm)
    ref = oracle.deep_train(X, Y, P, D, h, L, B, lr, E, perm=perm)
    assert ref["steps"] == 16 and len(gsl) == 16
    P0 = P.astype(np.float64)
    assert rel(gP - P0, ref["P"] - P0) <= 1e-3
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-3 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-3 * ref["epoch_loss"])


def test_train_eight_layers(mlp):
    """The deepest net the API takes (L = 8, h = 64), two shuffled epochs of
    1500 rows at batch 256 (tail of 220) on the evaluation recipe. The oracle
    itself moves by under 1e-6 when W0 is perturbed by 1e-7, so the bars are
    those of the one-layer path."""
    h, L, B, lr, E = 64, 8, 256, 0.002, 2
    d = datagen.make_data(1500, 32, epochs=E, seed=1005)
    P = _gauss_net(np.random.default_rng(9), h, L)
    gP, gsl, gel = _train(mlp, d.X, d.Y, P, h, L, B, lr, E, perm=d.perm)
    ref = oracle.deep_train(d.X, d.Y, P, D, h, L, B, lr, E, perm=d.perm)
    assert ref["steps"] == 12 and len(gsl) == 12
    P0 = P.astype(np.float64)
    assert rel(gP - P0, ref["P"] - P0) <= 1e-3
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-4 * ref["step_loss"])
    assert np.all(np.abs(gel - ref["epoch_loss"]) <= 1e-4 * ref["epoch_loss"])


def test_train_gaussian_workload_batch(mlp):
    """Three SGD steps of a 32-256-256-256-1 net at batch 4096 on the evaluation
    recipe (He-normal weights, sin target), against the oracle."""
    h, L, B, lr = 256, 3, 4096, 0.002
    d = datagen.make_data(20000, 32, epochs=1, seed=1005)
    P = _gauss_net(np.random.default_rng(7), h, L)
    gP, gsl, _ = _train(mlp, d.X, d.Y, P, h, L, B, lr, 1, perm=d.perm, max_steps=3)
    ref = oracle.deep_train(d.X, d.Y, P, D, h, L, B, lr, 1, perm=d.perm, max_steps=3)
    P0 = P.astype(np.float64)
    assert rel(gP - P0, ref["P"] - P0) <= 1e-3
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-4 * ref["step_loss"])


def test_zero_learning_rate(mlp):
    """lr = 0: the parameters stay bitwise as they were through a shuffled epoch
    (four steps, the last one a tail) and every step's loss is the batch MSE at
    the initial parameters, as the oracle's run with lr = 0 gives it."""
    h, L, B = 256, 2, 1000
    d = datagen.make_data(3400, 32, epochs=1, seed=77)
    P = _gauss_net(np.random.default_rng(77), h, L)
    gP, gsl, gel = _train(mlp, d.X, d.Y, P, h, L, B, 0.0, 1, perm=d.perm)
    assert np.array_equal(gP, P)
    ref = oracle.deep_train(d.X, d.Y, P, D, h, L, B, 0.0, 1, perm=d.perm)
    assert ref["steps"] == 4 and len(gsl) == 4
    assert np.all(np.abs(gsl - ref["step_loss"]) <= 1e-5 * ref["step_loss"])
    assert abs(gel[0] - ref["epoch_loss"][0]) <= 1e-5 * ref["epoch_loss"][0]


def test_deterministic(mlp):
    rng = np.random.default_rng(3)
    d = datagen.make_data(3000, 32, epochs=2, seed=8)
    P = _gauss_net(rng, 128, 3)
    a = _train(mlp, d.X, d.Y, P, 128, 3, 500, 0.01, 2, perm=d.perm)
    b = _train(mlp, d.X, d.Y, P, 128, 3, 500, 0.01, 2, perm=d.perm)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# --- errors --------------------------------------------------------------------

def test_errors(mlp):
    rng = np.random.default_rng(4)
    P = _gauss_net(rng, 64, 2)
    ctx, p = _ctx(mlp, P, 64, 2, 64)
    X = _to(rng.standard_normal((100, D)).astype(np.float32))
    Y = _to(rng.standard_normal(100).astype(np.float32))
    idx = np.arange(64, dtype=np.int32)
    idx[9] = 100                                      # one past the end: read as row 0, flagged
    mlp.mlp_deep_backward(ctx, X, Y, _to(idx))
    with pytest.raises(mlp.MLPError) as ei:
        mlp.mlp_deep_check_errors(ctx)
    assert ei.value.status == -6
    mlp.mlp_deep_check_errors(ctx)
    lib = mlp.load()
    before = p.clone()
    assert lib.mlp_deep_sgd_step(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 65,
                                 0.1, None) == -1           # B > max_batch
    assert lib.mlp_deep_sgd_step(ctx.handle, X.data_ptr(), 100, Y.data_ptr(), None, 10,
                                 float("nan"), None) == -1
    assert lib.mlp_deep_train_epochs(ctx.handle, X.data_ptr(), Y.data_ptr(), 100, 0, 0.1, 1,
                                     None, -1, None, None) == -1
    torch.cuda.synchronize()
    assert torch.equal(before, p)


def test_divergence_is_flagged(mlp):
    """As in the one-layer path: a learning rate of 1e30 overflows the next
    batch loss and mlp_deep_check_errors reports MLP_ERR_NONFINITE once."""
    h, L = 64, 2
    d = datagen.make_data(1024, 32, epochs=1, seed=72)
    P = _gauss_net(np.random.default_rng(72), h, L)
    ctx, _ = _ctx(mlp, P, h, L, 256)
    mlp.mlp_deep_train_epochs(ctx, _to(d.X), _to(d.Y), 256, 1e30, 1, perm=_to(d.perm))
    with pytest.raises(mlp.MLPError) as e:
        mlp.mlp_deep_check_errors(ctx)
    assert e.value.status == -5
    mlp.mlp_deep_check_errors(ctx)
