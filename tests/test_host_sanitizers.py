"""The host side of the library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The table builders (quadrature, real-basis mixing, operand words, entry lists),
the argument checks and the upload routine index many variable-length lists; a
copy of the library whose host code is compiled with both sanitizers
(build.build_sanitized: -Xarch_host -fsanitize=address,undefined, errors fatal)
runs the whole host test file in a child process with the sanitizer runtime
preloaded.  Leak detection is off: the Python interpreter itself keeps memory
until exit.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_host_tests_pass_under_sanitizers():
    from paper_2607_01408_amd import build

    lib = build.build_sanitized()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": build.sanitizer_runtime(),
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "SPINGTP_LIBRARY": lib,
    })
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"), "-q", "-x",
                        "-p", "no:cacheprovider", "-m", "not gpu"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=1500)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail
