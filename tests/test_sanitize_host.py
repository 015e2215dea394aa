"""CPU test job under AddressSanitizer + UndefinedBehaviorSanitizer.

Builds the sanitized oracle and the sanitized host half of the HIP library
(paper_2608_20532_amd/_build_sanitize.py), then runs the rest of the CPU suite in a
child Python process with clang's sanitizer runtime preloaded and both libraries
swapped in (F2ORACLE_LIB, F2GPU_LIB).  A first child call writes past a buffer
through the sanitized oracle and must be stopped by the sanitizer, so a green run
is known to have had the checks live."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(os.environ.get("F2_UNDER_SANITIZER") == "1", reason="already inside the job")


def _env(lib, orc):
    from paper_2608_20532_amd import _build_sanitize as B
    env = dict(os.environ)
    env.update(LD_PRELOAD=B.runtime(), F2GPU_LIB=lib, F2ORACLE_LIB=orc, F2_UNDER_SANITIZER="1",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", PYTHONDONTWRITEBYTECODE="1")
    return env


def test_cpu_suite_under_sanitizers():
    sys.path.insert(0, ROOT)
    from paper_2608_20532_amd import _build_sanitize as B
    lib, orc = B.build()
    env = _env(lib, orc)
    # the checks are live: an output buffer one word short is written past by the oracle
    probe = ("import numpy as np, oracle, ctypes\n"
             "L = oracle.lib(); assert 'san' in oracle._SO\n"
             "rows = np.array([[1, 5, 0], [0, 0, 0]], np.uint64); basis = np.zeros(2, np.uint64)\n"
             "piv = np.zeros(2, np.int32); M = np.zeros(4, np.uint64); nc = np.zeros(1, np.int32); fc = np.zeros(1, np.int64)\n"
             "p = lambda a: ctypes.c_void_p(a.ctypes.data)\n"
             "L.oracle_fit_context(p(rows), 2, 1, p(basis), p(piv), p(M), p(nc), p(fc))\n")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr, r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "tests", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0 and " passed" in r.stdout, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
