"""The multi-core oracle (oracle/oracle_mt.c) against the single-thread one.

It cuts every batch into 64 fixed row chunks and sums their partials in chunk
order, so its sums are reassociated: gradients, losses and trained weights may
differ from oracle.c by rounding only (held to 1e-13 relative here, against
about 1e-15 observed), the forward pass (no sum across rows) not at all, and no
result may depend on the number of threads."""
import numpy as np
import pytest

import datagen
import oracle


def _relmax(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


@pytest.mark.parametrize("h", [32, 256, 1024])
def test_forward_bitwise_equal(h):
    d = datagen.make_data(3000, h, seed=300 + h, with_perm=False)
    idx = np.random.default_rng(h).integers(0, 3000, size=2500).astype(np.int32)
    assert np.array_equal(oracle.mt_forward(d.X, d.W1, d.W2, idx=idx),
                          oracle.forward(d.X, d.W1, d.W2, idx=idx))
    assert np.array_equal(oracle.mt_forward(d.X, d.W1, d.W2), oracle.forward(d.X, d.W1, d.W2))


@pytest.mark.parametrize("h,B", [(256, 4096), (256, 63), (1024, 1000), (32, 1), (64, 65)])
def test_grad_matches_single_thread(h, B):
    d = datagen.make_data(5000, h, seed=310 + h + B, with_perm=False)
    idx = np.random.default_rng(B).integers(0, 5000, size=B).astype(np.int32)
    r1, r2, rl = oracle.grad(d.X, d.Y, d.W1, d.W2, idx=idx)
    m1, m2, ml = oracle.mt_grad(d.X, d.Y, d.W1, d.W2, idx=idx)
    assert _relmax(m1, r1) <= 1e-13 and _relmax(m2, r2) <= 1e-13
    assert abs(ml - rl) <= 1e-13 * rl


@pytest.mark.parametrize("k", [0, 1, 4])
def test_ten_steps_match_single_thread(k):
    w = datagen.WORKLOADS[k]
    n = min(w.n, 60000)
    d = datagen.make_data(n, w.hidden, epochs=1, shuffle=w.shuffle, seed=w.seed)
    ref = oracle.train(d.X, d.Y, d.W1, d.W2, w.batch, w.lr, 1, perm=d.perm, max_steps=10)
    got = oracle.mt_train(d.X, d.Y, d.W1, d.W2, w.batch, w.lr, 1, perm=d.perm, max_steps=10)
    assert got["steps"] == ref["steps"] == 10
    assert _relmax(got["W1"] - d.W1, ref["W1"] - d.W1) <= 1e-13
    assert _relmax(got["W2"] - d.W2, ref["W2"] - d.W2) <= 1e-13
    assert _relmax(got["step_loss"], ref["step_loss"]) <= 1e-13


def test_epochs_with_tail_and_identity_order():
    n, h, B, E, lr = 1000, 256, 64, 3, 0.01
    d = datagen.make_data(n, h, epochs=E, shuffle=True, seed=77)
    for perm in (d.perm, None):
        ref = oracle.train(d.X, d.Y, d.W1, d.W2, B, lr, E, perm=perm)
        got = oracle.mt_train(d.X, d.Y, d.W1, d.W2, B, lr, E, perm=perm)
        assert got["steps"] == ref["steps"] == 48
        assert _relmax(got["W1"], ref["W1"]) <= 1e-13
        assert _relmax(got["epoch_loss"], ref["epoch_loss"]) <= 1e-13


def test_thread_count_does_not_change_results():
    d = datagen.make_data(20000, 256, epochs=1, shuffle=True, seed=5)
    runs = []
    prev = oracle.mt_set_threads(1)
    try:
        for t in (1, 3, 8):
            oracle.mt_set_threads(t)
            runs.append(oracle.mt_train(d.X, d.Y, d.W1, d.W2, 1024, 0.005, 1, perm=d.perm,
                                        max_steps=6))
    finally:
        oracle.mt_set_threads(prev)
    for r in runs[1:]:
        assert np.array_equal(r["W1"], runs[0]["W1"]) and np.array_equal(r["W2"], runs[0]["W2"])
        assert np.array_equal(r["step_loss"], runs[0]["step_loss"])
