"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

A copy of the library is built with both sanitizers on its host code (the device code is
built as for the library) together with a C driver, tests/sanitize/abi_driver.cpp, that calls
every entry point of include/paraanya.h. Any out-of-bounds access, use after free, leak of the
library's own host memory or undefined behaviour in the host code ends the driver with a
sanitizer report and a non-zero status.
  * without a GPU: every argument check, NULL handle, status string, the allocation-free
    entry point's limits, and a valid create that fails at its first HIP call and must leave
    nothing behind;
  * on a GPU: additionally full samples through every entry point (linear and patch-MLP,
    one and two samples, split outputs, step noise, the allocation-free sample twice, the
    Parareal sampler) and a create that runs out of device memory.
"""
import os
import subprocess

import pytest

from paper_2609_36522_amd import build as B

SUPP = os.path.join(os.path.dirname(__file__), "sanitize", "lsan.supp")


def _driver():
    # Built by __graft_entry__.build(); built here only where nothing is (CPU runs).
    if not (os.path.exists(B.SAN_DRIVER) and os.path.exists(B.SAN_LIB)):
        B.build(sanitized=True)
    return B.SAN_DRIVER


def _run(mode, timeout):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:halt_on_error=1:abort_on_error=0:exitcode=23"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["LSAN_OPTIONS"] = f"suppressions={SUPP}:exitcode=23"
    r = subprocess.run([_driver(), mode], capture_output=True, text=True, timeout=timeout, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "abi_driver ok" in r.stdout, out[-4000:]
    assert "Sanitizer" not in out and "runtime error" not in out, out[-4000:]
    return out


def test_sanitized_abi_checks_without_gpu():
    out = _run("cpu", 300)
    assert "cpu checks ok" in out
    # The host code of the copy is instrumented (it imports the sanitizer runtime's hooks,
    # which the driver's executable provides).
    blob = open(B.SAN_LIB, "rb").read()
    assert b"__asan_report_load8" in blob and b"__ubsan_handle_" in blob


@pytest.mark.gpu
def test_sanitized_abi_full_runs():
    out = _run("gpu", 300)
    for line in ("linear, two samples ok", "patch-MLP, one sample ok", "patch-MLP, split outputs ok",
                 "allocation-free sample ok", "parareal ok", "out-of-memory create ok"):
        assert line in out, out[-4000:]
