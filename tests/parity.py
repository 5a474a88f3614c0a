"""Comparison helpers for GPU-vs-oracle parity (test infrastructure).

Relative error is normwise: ||a - ref||_F / ||ref||_F (rel). Next to it every
check also computes the largest elementwise error against the largest
reference entry, max|a - ref| / max|ref| (relmax), so that a few entries far
off cannot hide under a small normwise error; check() reports both and holds
both to the bar.

ReLU kink: where a pre-activation Z1[i, j] is so close to zero that fp32
cannot resolve its sign, both mask values are correct results of eq. (17).
The device computes Z1 as a length-32 dot product of fp32 values whose
products are formed from three-part bf16 splits on the matrix cores: each
product is within 2u |X_ik W1_kj| of exact (the dropped part products) and the
fp32 accumulation of the 6 x 32 part products adds at most gamma_38 ~ 38 u of
sum_k |X_ik W1_kj| (u = 2^-24), so the computed value differs from the exact
one by at most 40 u sum_k |X_ik W1_kj|; 41 u is used. (A plain fp32 dot product
would need gamma_32 ~ 32 u.) Entries with |Z1| under that bound are ambiguous. Before dW1 is
compared, each column's ambiguous rows are resolved by choosing the subset of
their contributions X_i * g_i * W2_j (g_i = (2/n_b)(Ypred_i - Y_i)) that best
matches the GPU column, by brute force over subsets (at most 2^10). dW2, Ypred
and the loss are continuous at the kink and need no alignment.
"""
import itertools

import numpy as np

U32 = 2.0 ** -24
KINK_GAMMA = 41 * U32


def rel(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(a - ref) / (den if den > 0 else 1.0))


def relmax(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    return float(np.max(np.abs(a - ref)) / (den if den > 0 else 1.0)) if ref.size else 0.0


def check(name, a, ref, bar):
    """Assert rel(a, ref) <= bar and relmax(a, ref) <= bar; print both."""
    e, m = rel(a, ref), relmax(a, ref)
    print("%-24s rel %.3e  relmax %.3e  (bar %.0e)" % (name, e, m, bar), flush=True)
    assert e <= bar, (name, "normwise", e, bar)
    assert m <= bar, (name, "max elementwise", m, bar)
    return e, m


def align_kinks(dW1_gpu, dW1_ref, X, Y, W1, W2, idx, z, zabs, ypred):
    """Return (dW1_ref adjusted to the GPU's choice at ambiguous entries,
    number of ambiguous entries, number of flips accepted)."""
    nb = z.shape[0]
    rows = np.arange(nb) if idx is None else np.asarray(idx)
    Xb = X[rows].astype(np.float64)
    g = (2.0 / nb) * (ypred - Y[rows].astype(np.float64))
    amb = np.abs(z) <= KINK_GAMMA * zabs
    out = dW1_ref.copy()
    n_amb = int(amb.sum())
    flips = 0
    for j in np.nonzero(amb.any(axis=0))[0]:
        ii = np.nonzero(amb[:, j])[0]
        if len(ii) > 10:
            raise AssertionError("too many ambiguous kink entries in column %d" % j)
        contrib = Xb[ii] * (g[ii] * W2[j])[:, None]          # [m, d]
        on = z[ii, j] > 0
        base = dW1_ref[:, j] - contrib[on].sum(axis=0)
        best, best_err, best_sel = None, np.inf, None
        for sel in itertools.product((False, True), repeat=len(ii)):
            sel = np.array(sel)
            cand = base + contrib[sel].sum(axis=0)
            err = np.linalg.norm(cand - dW1_gpu[:, j])
            if err < best_err:
                best, best_err, best_sel = cand, err, sel
        out[:, j] = best
        flips += int((best_sel != on).sum())
    return out, n_amb, flips


def loss_tolerance(loss_ref, z, zabs, W2, rel_bar=1e-5):
    """Bar for the batch MSE computed in fp32.

    Ypred_i = sum_j ReLU(Z1_ij) W2_j carries an fp32 rounding error
    delta_i <~ 4 sqrt(h + 32) u S_i (random-walk bound), with
    S_i = sum_j |ReLU(Z1_ij) W2_j| + |W2_j| sum_k |X_ik W1_kj|. The loss
    L = mean(r_i^2) then moves by about 2 sqrt(L) rms(delta): when Ypred is close
    to Y (a cancellation in r_i) this absolute term, not the relative one, is the
    honest bound."""
    W2 = np.abs(np.reshape(W2, -1))
    h = z.shape[1]
    S = np.maximum(z, 0.0) @ W2 + zabs @ W2
    delta = 4.0 * np.sqrt(h + 32.0) * U32 * S
    return rel_bar * loss_ref + 2.0 * np.sqrt(loss_ref) * np.sqrt(np.mean(delta ** 2))
