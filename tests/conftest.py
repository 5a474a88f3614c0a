import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionfinish(session, exitstatus):
    """In the sanitized run (tests/test_host_sanitizers.py), list the instrumented
    libraries this process mapped, so the parent can check they were used."""
    if os.environ.get("MLP_SANITIZED_RUN") != "1":
        return
    want = [os.environ.get("ORACLE_LIBDIR", ""), os.environ.get("MLP_LIBRARY", "")]
    seen = set()
    with open("/proc/self/maps") as f:
        for line in f:
            path = line.split()[-1] if len(line.split()) >= 6 else ""
            if any(w and path.startswith(w) for w in want):
                seen.add(path)
    for p in sorted(seen):
        print("\n[sanitized run] loaded " + p)
