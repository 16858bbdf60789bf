"""The host-only ABI checks of test_abi_cpu.py once more, against a build of the
library whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer
(device code unchanged; nothing here launches a kernel). The ASan runtime is
preloaded into a child Python; any sanitizer report fails the test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_pass_under_asan_and_ubsan(tmp_path):
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("this process already has a preload, which the sanitizer runtime would replace")
    from paper_2601_08670_amd import build_sanitized as S
    lib = S.build(str(tmp_path))
    rt = S.runtime()
    assert os.path.exists(rt), rt
    env = dict(os.environ, LD_PRELOAD=rt, PCED_LIBRARY=lib, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"), "-q",
                        "-p", "no:cacheprovider"], env=env, capture_output=True, text=True, timeout=900, cwd=ROOT)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out and " failed" not in out
