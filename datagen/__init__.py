"""Seeded synthetic inputs for the 32-h-1 ReLU/MSE regression workloads.

This module only draws numbers. It holds none of the training arithmetic, so
both the fp64 oracle and the HIP path can consume its arrays without sharing
any part of the method.

The paper trains a 32-256-1 network with no biases (Sec. III.A, eq. 10) on a
dataset it does not describe (Sec. VI.A). The stand-in is a smooth noisy
regression target over Gaussian inputs:

    a  ~ N(0, 1/32)            (variance 1/32)         shape [32]
    X  ~ N(0, 1)               drawn fp64, stored fp32 shape [n, 32]
    Y  = fp32( sin(X . a) + 0.1 * N(0, 1) )            shape [n]
    W1 = fp32( N(0, 1) * sqrt(2/32) )   He-normal      shape [32, h]
    W2 = fp32( N(0, 1) * sqrt(2/h) )    He-normal      shape [h]
    perm_e = permutation of [0, n) per epoch (int32), or identity order

Draw order is fixed: one SeedSequence(seed) spawns five PCG64 child streams,
used in this order: a, X, noise, W, perm. X is drawn in chunks of 2^20 rows;
the stream is order preserving, so the chunking does not change the values.
Y is computed from the fp32-rounded X promoted to fp64, so it is a function
of the inputs the network actually sees.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

D_IN = 32
_CHUNK = 1 << 20


@dataclasses.dataclass(frozen=True)
class Workload:
    """One training workload: a d-h-1 net, n samples, mini-batch SGD."""
    name: str
    hidden: int
    n: int
    batch: int
    lr: float
    epochs: int
    shuffle: bool
    seed: int
    d_in: int = D_IN
    layers: int = 1            # hidden layers of width `hidden`

    @property
    def steps_per_epoch(self) -> int:
        return -(-self.n // self.batch)

    @property
    def steps(self) -> int:
        return self.steps_per_epoch * self.epochs

    @property
    def tail(self) -> int:
        """Rows in the last batch of an epoch (== batch when n % batch == 0)."""
        r = self.n % self.batch
        return r if r else self.batch

    @property
    def samples(self) -> int:
        return self.n * self.epochs

    def flop_per_sample(self) -> int:
        """Contractions of one SGD step per sample at 2 FLOP per multiply-add.
        One hidden layer: 2*(d*h + h + h + h + d*h) (Z1, Ypred, dW2, dZ1, dW1).
        L layers: forward d*h + (L-1)*h^2 + h, weight gradients the same, the
        output's back-propagation h, and (L-1)*h^2 for the hidden dH."""
        d, h, L = self.d_in, self.hidden, self.layers
        fwd = d * h + (L - 1) * h * h + h
        return 2 * (2 * fwd + h + (L - 1) * h * h)


# The five evaluation workloads. Their seeds are 1000 + k for workload k.
WORKLOADS = [
    Workload("mlp32-256-1_n1024_b64_e5", 256, 1024, 64, 0.01, 5, False, 1001),
    Workload("mlp32-256-1_n100k_b256_e10", 256, 100_000, 256, 0.01, 10, True, 1002),
    Workload("mlp32-256-1_n1M_b1024_e10", 256, 1_000_000, 1024, 0.005, 10, True, 1003),
    Workload("mlp32-1024-1_n1M_b1024_e5", 1024, 1_000_000, 1024, 0.005, 5, True, 1004),
    Workload("mlp32-256-1_n10M_b4096_e3", 256, 10_000_000, 4096, 0.002, 3, True, 1005),
]

# The paper's hidden-width sweep (Sec. VI.C, Table II): n = 2,560 samples,
# batch 256, lr 0.002 and 100 epochs (the training setup of Sec. III.A), hidden
# width 32 ... 1024. The paper does not say whether batches are shuffled; these
# use a seeded per-epoch permutation like the evaluation workloads.
SWEEP_HIDDEN = (32, 64, 128, 256, 512, 1024)
SWEEP = [Workload("mlp32-%d-1_n2560_b256_e100" % h, h, 2560, 256, 0.002, 100, True, 2000 + h)
         for h in SWEEP_HIDDEN]

# The dataset sizes of the paper's strategy comparison (Sec. VI.B, Table I):
# 256, 2,560 and 25,600 samples of the 32-256-1 net, batch 256, lr 0.002,
# 100 epochs.
TABLE1 = [Workload("mlp32-256-1_n%d_b256_e100" % n, 256, n, 256, 0.002, 100, True, 3000 + i)
          for i, n in enumerate((256, 2560, 25600))]

# Deeper networks (the paper's future work, Sec. VII.B): L hidden layers of
# width h on the 1M-sample recipe, batch 4096, lr 0.002, one epoch.
DEEP = [Workload("mlp32-%sx%d-1_n1M_b4096_e1" % (h, L), h, 1_000_000, 4096, 0.002, 1, True,
                 4000 + 10 * L + h // 64, layers=L)
        for h, L in ((256, 2), (256, 3), (1024, 2))]

SUITES = {"configs": WORKLOADS, "sweep": SWEEP, "table1": TABLE1, "deep": DEEP}


@dataclasses.dataclass
class Data:
    X: np.ndarray      # [n, d] float32, row-major
    Y: np.ndarray      # [n] float32
    W1: np.ndarray     # [d, h] float32, row-major (rows = inputs)
    W2: np.ndarray     # [h] float32
    perm: np.ndarray | None   # [epochs, n] int32, or None for identity order
    a: np.ndarray      # [d] float64 target direction (data recipe only)


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(5)]


def make_data(n: int, hidden: int, epochs: int = 1, shuffle: bool = True,
              seed: int = 0, d_in: int = D_IN, with_perm: bool = True) -> Data:
    """Draw X, Y, W1, W2 and the per-epoch permutations for one workload."""
    if n < 0 or hidden <= 0 or d_in <= 0 or epochs < 0:
        raise ValueError("bad sizes")
    r_a, r_x, r_noise, r_w, r_perm = _streams(seed)
    a = r_a.standard_normal(d_in) / math.sqrt(d_in)
    X = np.empty((n, d_in), dtype=np.float32)
    Y = np.empty(n, dtype=np.float32)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        X[s:e] = r_x.standard_normal((e - s, d_in))
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        t = X[s:e].astype(np.float64) @ a
        Y[s:e] = np.sin(t) + 0.1 * r_noise.standard_normal(e - s)
    W1 = (r_w.standard_normal((d_in, hidden)) * math.sqrt(2.0 / d_in)).astype(np.float32)
    W2 = (r_w.standard_normal(hidden) * math.sqrt(2.0 / hidden)).astype(np.float32)
    perm = None
    if with_perm and shuffle and epochs > 0:
        perm = np.empty((epochs, n), dtype=np.int32)
        for e in range(epochs):
            perm[e] = r_perm.permutation(n).astype(np.int32)
    return Data(X, Y, W1, W2, perm, a)


def make_workload(w: Workload, n: int | None = None) -> Data:
    """Inputs for workload ``w``; ``n`` overrides the sample count (same recipe)."""
    return make_data(w.n if n is None else n, w.hidden, w.epochs, w.shuffle, w.seed, w.d_in)


def make_deep_params(d_in: int, hidden: int, layers: int, seed: int) -> np.ndarray:
    """He-normal parameters of a d_in-h-...-h-1 net in one flat fp32 array:
    W_1 [d_in x h] (std sqrt(2/d_in)), W_2 .. W_L [h x h] (std sqrt(2/h)), then
    w_o [h] (std sqrt(2/h))."""
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    parts = []
    for l in range(layers):
        fan_in = d_in if l == 0 else hidden
        parts.append(r.standard_normal(fan_in * hidden) * math.sqrt(2.0 / fan_in))
    parts.append(r.standard_normal(hidden) * math.sqrt(2.0 / hidden))
    return np.concatenate(parts).astype(np.float32)


def identity_perm(epochs: int, n: int) -> np.ndarray:
    return np.broadcast_to(np.arange(n, dtype=np.int32), (epochs, n)).copy()
