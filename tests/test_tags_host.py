"""Host arithmetic of the trainer's step tags (paper_2606_30497_amd/csrc/tags.h),
compiled with g++ (under ASan and UBSan) on the CPU: a launch never uses tag 0, never uses a tag range
that wraps past 2^32, the next launch starts past every tag of this one, and a
range that would wrap restarts at 1 with the exchange words cleared."""
import os
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_30497_amd", "csrc")

DRIVER = r"""
#include <stdio.h>
#include <stdlib.h>
#include "tags.h"
int main(int argc, char **argv) {
    for (int i = 1; i + 1 < argc; i += 2) {
        const unsigned long long base = strtoull(argv[i], 0, 10);
        const long long steps = strtoll(argv[i + 1], 0, 10);
        const mlp::TagPlan p = mlp::plan_tags((uint32_t)base, steps);
        printf("%u %u %d\n", p.base, p.next, p.clear ? 1 : 0);
    }
    return 0;
}
"""

CASES = [(1, 10), (1, (1 << 30) - 1), (12345, 7326), (0, 5),
         (0xFFFFFFFF - 12, 10), (0xFFFFFFFF - 12, 11), (0xFFFFFFFF - 12, 12),
         (0xFFFFFFFF, 1), (0xFFFFFFFF - (1 << 30), (1 << 30) - 1), (0x80000000, 1 << 29)]


@pytest.fixture(scope="module")
def driver():
    d = tempfile.mkdtemp()
    src = os.path.join(d, "tags_driver.cpp")
    exe = os.path.join(d, "tags_driver")
    with open(src, "w") as f:
        f.write(DRIVER)
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-Wall", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", "-I" + CSRC, src, "-o", exe],
                          env=_env())
    return exe


def _env():
    # the driver carries its own sanitizer runtime: no preloaded one from a parent
    return {k: v for k, v in os.environ.items() if k != "LD_PRELOAD"}


def _plans(driver, cases):
    args = [str(x) for c in cases for x in c]
    out = subprocess.check_output([driver] + args, text=True, env=_env()).split("\n")
    return [tuple(int(v) for v in line.split()) for line in out if line.strip()]


def test_tag_ranges(driver):
    for (base, steps), (b, nxt, clear) in zip(CASES, _plans(driver, CASES)):
        # the launch's tags b .. b + steps - 1 are nonzero and do not wrap
        assert b >= 1 and b + steps - 1 <= 0xFFFFFFFF, (base, steps)
        # the next launch starts past them (a gap of two), without wrapping
        assert nxt == b + steps + 2 <= 0xFFFFFFFF, (base, steps)
        # a base kept unless it is 0 or its range would wrap; otherwise restart at 1, cleared
        keep = base >= 1 and base + steps + 2 <= 0xFFFFFFFF
        assert (b, clear) == ((base, 0) if keep else (1, 1)), (base, steps)


def test_many_launches_never_reuse_a_live_tag(driver):
    """A context's launches in sequence: every launch's range lies past the
    previous one's unless the words were cleared in between."""
    base, prev_end = 0xFFFFFFFF - 100000, None
    seq = [7326, 80, 50000, 3, 9770, 40000, 1, 1]
    for steps in seq:
        (b, nxt, clear), = _plans(driver, [(base, steps)])
        if prev_end is not None and not clear:
            assert b > prev_end + 1
        prev_end = b + steps - 1
        base = nxt
