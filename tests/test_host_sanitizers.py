"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/host_checks/build.py builds a copy of libhv whose host code carries
both sanitizers (device code as usual) and links tests/host_checks/host_checks.c
against it; the driver runs leaf layout, workspace and plan sizing, Merkle,
tree and stream-batch planning over thousands of seeded random message sets,
and every entry point's argument checks, all on the host (nothing it calls
reaches a GPU).  Any sanitizer report ends the run with a failure.
"""
import importlib.util
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _builder():
    """tests/host_checks/build.py, loaded by path under a name of its own."""
    spec = importlib.util.spec_from_file_location("hv_host_checks_build", os.path.join(HERE, "host_checks", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.timeout(900)
def test_host_code_is_clean_under_sanitizers():
    exe = _builder().build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.strip().splitlines()[-1] == "host checks passed", r.stdout[-2000:]
