"""Plant plausible mistakes in copies of oracle_deep.c and check that the pins
of tests/test_oracle_deep_pins.py reject each one.

Every mutant is a text edit compiled into a temporary library; the original
source is never touched."""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_deep_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle_deep.c")

MUTANTS = {
    "relu_prime_zero_is_one": ("b.dh[j] = z[j] > 0.0 ? b.dh[j] : 0.0;",
                               "b.dh[j] = z[j] >= 0.0 ? b.dh[j] : 0.0;"),
    "no_relu_mask_in_backward": ("b.dh[j] = z[j] > 0.0 ? b.dh[j] : 0.0;", "b.dh[j] = b.dh[j];"),
    "scale_one_over_n": ("const double scale = 2.0 / (double)nb;",
                         "const double scale = 1.0 / (double)nb;"),
    "forward_weights_transposed": ("double p = hp[k] * W[(int64_t)k * h + j];",
                                   "double p = hp[k] * W[(int64_t)j * K + k];"),
    "dw_transposed": ("dW[(int64_t)k * h + j] += hp[k] * b.dh[j];",
                      "dW[(int64_t)j * K + k] += hp[k] * b.dh[j];"),
    "backprop_without_transpose": ("acc += b.dh[j] * W[(int64_t)k * h + j];",
                                   "acc += b.dh[j] * W[(int64_t)j * h + k];"),
    "dh_not_propagated": ("memcpy(b.dh, b.dhn, sizeof(double) * (size_t)K);", ""),
    "dw_uses_layer_output": ("const double *hp = b.hin + (size_t)(l - 1) * b.w;\n"
                             "            const double *z = b.z",
                             "const double *hp = b.hin + (size_t)l * b.w;\n"
                             "            const double *z = b.z"),
    "output_grad_without_wo": ("b.dh[j] = g * wo[j];", "b.dh[j] = g;"),
    "forward_without_relu": ("hn[j] = acc > 0.0 ? acc : 0.0;", "hn[j] = acc;"),
    "update_sign": ("P[i] -= lr * dP[i];", "P[i] += lr * dP[i];"),
    "tail_weighted_as_full": ("epoch_sse += Lb * (double)nb;", "epoch_sse += Lb * (double)batch;"),
}


def _pins():
    yield lambda: pins.test_one_layer_matches_the_shallow_oracle(8)
    yield lambda: pins.test_finite_differences(4, 6, 3, 1)
    yield lambda: pins.test_all_active_net_is_linear(3)
    yield lambda: pins.test_torch_autograd(64, 3)
    yield pins.test_relu_prime_at_zero_through_two_layers


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor missing or ambiguous: " + old
    path_c = tmp_path / "mutant.c"
    path_c.write_text(src.replace(old, new))
    path_so = tmp_path / ("liboracle_deep_%s.so" % name)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-o", str(path_so), str(path_c), "-lm"])
    caught = []
    with oracle.swapped_deep_library(str(path_so)):
        for pin in _pins():
            try:
                pin()
            except AssertionError:
                caught.append(pin)
    assert caught, "no pin rejects mutant " + name
