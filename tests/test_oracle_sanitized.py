"""The oracle's test files again with the oracle built under AddressSanitizer
and UndefinedBehaviorSanitizer (out-of-bounds accesses, use after free,
signed overflow, bad shifts in the 128/256-bit arithmetic abort the run), in
a child process that preloads the ASan runtime; the host-side input generator
runs there too.  CPU only."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_TESTS = ["test_oracle_golden.py", "test_oracle_bruteforce.py", "test_oracle_invariants.py",
                "test_oracle_special.py", "test_oracle_paper_table.py", "test_oracle_sharded.py",
                "test_oracle_adoption.py", "test_oracle_stats.py", "test_oracle_join.py"]


def _runtime():
    try:
        p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    except OSError:
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.skipif(_runtime() is None, reason="no gcc AddressSanitizer runtime")
def test_oracle_suite_under_asan_and_ubsan():
    env = dict(os.environ, ATREX_ORACLE_SANITIZE="1", LD_PRELOAD=_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    build = subprocess.run([sys.executable, "-c",
                            "from oracle import oracle as O; O.build(force=True); O.lib(); print(O.library_path())"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-3000:]
    assert build.stdout.strip().endswith("libatrex_oracle_san.so"), build.stdout
    run = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          *[os.path.join("tests", f) for f in ORACLE_TESTS]],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    tail = (run.stdout + run.stderr)[-4000:]
    assert run.returncode == 0, tail
    assert "passed" in run.stdout and "ERROR: AddressSanitizer" not in run.stderr, tail
