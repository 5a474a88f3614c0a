"""The CPU test suite again, with every host library built under AddressSanitizer
and UndefinedBehaviorSanitizer: the three oracle libraries (oracle.c,
oracle_deep.c, oracle_mt.c) and the host code of libmlp.so (the C ABI's
argument checks, sizing and context handling; the device code is unchanged).

Both are built with the ROCm clang, so that one sanitizer runtime serves the
process: it is preloaded into a child pytest run of every other CPU test, which
loads the instrumented copies through ORACLE_LIBDIR and MLP_LIBRARY. The run
runs without output capture (a sanitizer stops the process, and its report
must not stay in a captured buffer); it must pass, print no sanitizer report, and have mapped both instrumented
libraries (the child's conftest lists what it loaded). Leak checking is off:
the interpreter itself does not free everything at exit.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LLVM = "/opt/rocm/llvm"
CLANG = os.path.join(LLVM, "bin", "clang")


def _runtime():
    hits = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    return hits[-1] if hits else None


pytestmark = pytest.mark.skipif(
    os.environ.get("MLP_SANITIZED_RUN") == "1" or not os.path.exists(CLANG) or _runtime() is None,
    reason="inside the sanitized run itself, or no ROCm clang / sanitizer runtime")


def test_cpu_suite_clean_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    import oracle
    from paper_2606_30497_amd import build as mlp_build

    rt = _runtime()
    rtdir = os.path.dirname(rt)
    odir = tmp_path / "oracle"
    odir.mkdir()
    oracle.build(out_dir=str(odir), cc=CLANG,
                 extra=("-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                        "-fno-omit-frame-pointer", "-g", "-shared-libsan",
                        "-Wl,-rpath," + rtdir, "-Wl,-rpath," + os.path.join(LLVM, "lib")))
    lib = str(tmp_path / "libmlp_san.so")
    host = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize=vptr",
              "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"):
        host += ["-Xarch_host", f]
    mlp_build.build(out=lib, build_dir=str(tmp_path / "obj"), extra=host)

    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, MLP_SANITIZED_RUN="1", ORACLE_LIBDIR=str(odir),
               MLP_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "tests", "-x", "-q", "-m", "not gpu",
                        "-s", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=900)
    out = r.stdout
    tail = "\n".join(out.splitlines()[-40:])
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in out and "runtime error:" not in out, tail
    loaded = [l for l in out.splitlines() if l.startswith("[sanitized run] loaded ")]
    paths = " ".join(loaded)
    for name in ("liboracle.so", "liboracle_deep.so", "liboracle_mt.so"):
        assert os.path.join(str(odir), name) in paths, (name, loaded)
    assert lib in paths, loaded
