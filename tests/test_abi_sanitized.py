"""The C ABI's host code (argument validation, planning, the staging pool,
launch set-up) under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds libapack with its host code sanitized (the device code is compiled as
in the product build) and runs the CPU-only ABI tests against it in a child
process that preloads the sanitizer runtime; any report fails the run.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_tests_pass_under_address_and_ub_sanitizers(tmp_path):
    from paper_2608_08794_amd import build as B
    try:
        runtime = B.asan_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = B.build_sanitized()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": runtime,
        "APACK_LIBRARY": lib,
        "ASAN_OPTIONS": f"detect_leaks=0:halt_on_error=1:log_path={tmp_path}/asan",
        "UBSAN_OPTIONS": f"halt_on_error=1:print_stacktrace=1:log_path={tmp_path}/ubsan",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"), "-x", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    reports = sorted(p for p in os.listdir(tmp_path) if p.startswith(("asan", "ubsan")))
    text = "".join(open(os.path.join(tmp_path, p)).read()[:4000] for p in reports)
    assert r.returncode == 0 and not reports, (r.stdout[-3000:] + r.stderr[-3000:] + text)
