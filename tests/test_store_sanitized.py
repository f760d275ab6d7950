"""The host context store (context_store.cpp, plain C++) built alone with g++
under AddressSanitizer and UndefinedBehaviorSanitizer, with the store tests
run against it in a child process.  CPU only; skipped where g++ or the
sanitizer runtimes are missing."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

RUNNER = r"""
import ctypes, sys
sys.path.insert(0, {root!r})
from paper_2405_19888_amd import binding
lib = ctypes.CDLL({lib!r})
lib.parrot_last_error.argtypes = []
lib.parrot_last_error.restype = ctypes.c_char_p
binding._lib = lib
import pytest
sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", {tests!r}]))
"""


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_context_store_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("sanitizer runtimes not available")
    lib = str(tmp_path / "libstore_sanitized.so")
    src = os.path.join(ROOT, "paper_2405_19888_amd", "csrc", "context_store.cpp")
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined", "-shared", "-fPIC",
                    "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(ROOT, "paper_2405_19888_amd", "csrc"),
                    src, os.path.join(ROOT, "tests", "sanitizer_stub.cpp"), "-o", lib], check=True)
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}", ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    code = RUNNER.format(root=ROOT, lib=lib, tests=os.path.join(ROOT, "tests", "test_context_store.py"))
    p = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    assert p.returncode == 0, p.stdout[-3000:] + p.stderr[-3000:]
    assert "passed" in p.stdout
