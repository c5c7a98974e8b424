"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer.

oracle/selfcheck.c runs the oracle's pins in C (golden worked examples, the
integer rounding formula over a sweep of FP32 patterns, round trips and the
bookkeeping invariants of every function; its header lists them).  It is built
twice by oracle.build_selfcheck -- with the oracle's own optimisation, and with
-fsanitize=address,undefined (runtime linked statically into the executable,
any finding fatal) -- and both builds must pass every check.  A memory error or
undefined behaviour anywhere in the oracle on those inputs fails the sanitized
run.
"""
import os
import shutil
import subprocess

import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _run(sanitize: bool):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    try:
        exe = oracle.build_selfcheck(sanitize=sanitize)
    except subprocess.CalledProcessError as e:
        if sanitize:
            pytest.skip(f"sanitizer build failed (runtime missing?): {e}")
        raise
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe, GOLDEN], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "checks passed" in run.stdout
    assert int(run.stdout.split()[1]) > 17_000_000, run.stdout  # the cast sweep: 2^32 / 251


def test_selfcheck_plain():
    _run(sanitize=False)


def test_selfcheck_address_and_undefined_sanitizers():
    _run(sanitize=True)
