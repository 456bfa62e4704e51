"""The host ABI tests again, against the host-sanitized build of the library.

build.py --sanitize compiles the same sources with the host code (packer,
unpacker, argument validation, launch planning) instrumented by
AddressSanitizer and UndefinedBehaviorSanitizer, every finding fatal.  The
test runs tests/test_abi_host.py in a child process that loads that build
(Q4NX_LIBRARY) with clang's ASan runtime preloaded.  CPU only: the device
entry points are only reached with invalid arguments, which are rejected
before any HIP call.
"""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_06063_amd", "csrc")


def _build_module():
    spec = importlib.util.spec_from_file_location("q4nx_build", os.path.join(ROOT, "paper_2602_06063_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _stale(lib):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = [os.path.join(CSRC, f) for f in os.listdir(CSRC)] + [os.path.join(ROOT, "include", "q4nx.h")]
    return any(os.path.getmtime(s) > t for s in srcs)


def test_host_abi_under_asan_and_ubsan():
    b = _build_module()
    if not os.path.exists(b.hipcc()):
        pytest.skip("hipcc not available")
    lib = b.ASAN_LIB
    if _stale(lib):
        b.build(sanitize=True)
    env = dict(os.environ)
    env.update(Q4NX_LIBRARY=lib, LD_PRELOAD=b.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    # The child really loaded the sanitized build.
    assert " passed" in out
