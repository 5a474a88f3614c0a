"""Plant plausible mistakes in copies of the oracle and check the pins catch each.

Every mutant is a text edit of oracle.c compiled into a temporary library; the
original source is never touched. A mutant passes this test only when at least
one pin from test_oracle_pins.py fails against it.
"""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "relu_prime_zero_is_one": ("double dz1 = z[j] > 0.0 ?", "double dz1 = z[j] >= 0.0 ?"),
    "scale_one_over_n": ("const double scale = 2.0 / (double)nb;", "const double scale = 1.0 / (double)nb;"),
    "residual_sign": ("double res = y - (double)Y[r];", "double res = (double)Y[r] - y;"),
    "forward_w1_transposed": ("double p = (double)x[k] * W1[(int64_t)k * h + j];",
                              "double p = (double)x[k] * W1[(int64_t)j * d + k];"),
    "dw1_transposed": ("dW1[(int64_t)k * h + j] += (double)x[k] * dz1;",
                       "dW1[(int64_t)j * d + k] += (double)x[k] * dz1;"),
    "dw2_uses_z_not_h": ("dW2[j] += hj * g;", "dW2[j] += z[j] * g;"),
    "ypred_without_relu": ("y += (acc > 0.0 ? acc : 0.0) * W2[j];", "y += acc * W2[j];"),
    "update_sign": ("W1[i] -= lr * dW1[i];", "W1[i] += lr * dW1[i];"),
    "loss_divisor": ("if (loss) *loss = sse / (double)nb;", "if (loss) *loss = sse / (double)(nb + 1);"),
    "tail_weighted_as_full": ("epoch_sse += L * (double)nb;", "epoch_sse += L * (double)batch;"),
    "dz1_without_w2": ("double dz1 = z[j] > 0.0 ? g * W2[j] : 0.0;", "double dz1 = z[j] > 0.0 ? g : 0.0;"),
    "w2_update_dropped": ("for (int32_t j = 0; j < h; ++j) W2[j] -= lr * dW2[j];", ""),
}


def _pins():
    yield pins.test_worked_two_sample_step
    yield pins.test_relu_prime_at_zero_is_zero
    yield lambda: pins.test_finite_differences_4_8_1(0)
    yield lambda: pins.test_torch_autograd_real_shapes(32, 257)
    yield pins.test_torch_sgd_loop_with_shuffle_and_tail


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor missing: " + old
    path_c = tmp_path / "mutant.c"
    path_c.write_text(src.replace(old, new))
    path_so = tmp_path / ("liboracle_%s.so" % name)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-o", str(path_so), str(path_c), "-lm"])
    caught = []
    with oracle.swapped_library(str(path_so)):
        for pin in _pins():
            try:
                pin()
            except AssertionError:
                caught.append(pin)
    assert caught, "no pin rejects mutant " + name
