"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

oracle/sanitize_driver.c calls every oracle function on small seeded
inputs with buffers of exactly the documented sizes; built together with
oracle/gpic_oracle.c with -fsanitize=address,undefined (and the oracle's
own floating-point flags), any out-of-bounds access, use after free, leak
or undefined arithmetic ends the run with a report, and the driver's own
invariant checks must pass."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_ub_sanitizers():
    d = tempfile.mkdtemp(prefix="oracle_san_")
    try:
        exe = os.path.join(d, "sanitize_driver")
        cmd = ["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-fno-omit-frame-pointer",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               "-o", exe, os.path.join(ORACLE, "sanitize_driver.c"),
               os.path.join(ORACLE, "gpic_oracle.c"), "-lm"]
        b = subprocess.run(cmd, capture_output=True, text=True)
        assert b.returncode == 0, b.stderr
        # the build really carries both runtimes
        libs = subprocess.run(["ldd", exe], capture_output=True, text=True).stdout
        assert "libasan" in libs and "libubsan" in libs, libs
        env = dict(os.environ, OMP_NUM_THREADS="4",
                   ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr
        assert "all checks passed" in r.stdout
    finally:
        shutil.rmtree(d, ignore_errors=True)
