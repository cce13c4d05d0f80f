"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(runs without a GPU): tests/sanitize/abi_fuzz.c drives every C-ABI entry point
with seeded random, extreme and defective arguments against a build of the
library whose host pass is instrumented; every call must be rejected on the
host (never reach the device) or, for the pure host calls, give consistent
results, with no sanitizer report."""
import os
import subprocess

import pytest

from conftest import ROOT


def _exe():
    import importlib.util

    path = os.path.join(ROOT, "tests", "sanitize", "build.py")
    spec = importlib.util.spec_from_file_location("sanitize_build", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    if not os.path.exists(mod.EXE) or os.path.getmtime(mod.EXE) < os.path.getmtime(
            os.path.join(ROOT, "paper_1902_11208_amd", "libmdlstm.so")):
        mod.build()
    return mod.EXE


def test_host_validation_under_sanitizers(built_lib):
    try:
        exe = _exe()
    except RuntimeError as e:
        pytest.skip(f"sanitizer build unavailable: {e}")
    env = dict(os.environ)
    # no device is visible to the check, whatever machine it runs on
    env.update(HIP_VISIBLE_DEVICES="", ROCR_VISIBLE_DEVICES="", CUDA_VISIBLE_DEVICES="",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe, "20000"], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    print(r.stdout)
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert "0 failures" in r.stdout
