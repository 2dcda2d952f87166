"""The oracle's pins run again against an AddressSanitizer +
UndefinedBehaviorSanitizer build of the oracle library (every report aborts
the run), in a child process that preloads the ASan runtime."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# the pins of every oracle part; the KDE file's unbinned-density pins use
# numpy only and add nothing here
ORACLE_TESTS = ["test_oracle_summarize.py", "test_oracle_cross_rank.py", "test_oracle_l1.py", "test_oracle_kde.py",
                "test_oracle_w1.py", "test_oracle_l2.py", "test_oracle_compact.py"]


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.timeout(900)
def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's ASan runtime is not installed")
    sys.path.insert(0, ROOT)
    import oracle.build
    lib = oracle.build.build(out=str(tmp_path / "liboracle_san.so"), sanitize=True)
    env = dict(os.environ)
    env.update({
        "ARGUS_ORACLE_LIB": lib,
        "LD_PRELOAD": asan,
        # the interpreter itself is not instrumented: its allocations are not
        # leak-checked; every oracle report is fatal
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
           *[os.path.join(ROOT, "tests", t) for t in ORACLE_TESTS]]
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, tail
