"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer,
without a GPU: the library is built with host-side sanitizers and the ABI
tests that need no GPU run against it in a child process with the sanitizer
runtime preloaded.  Any sanitizer report aborts the child and fails the test."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(_asan_runtime() is None, reason="no ASan runtime in this ROCm")
def test_abi_checks_under_host_sanitizers(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2601_21473_amd.build import build
    lib = build(out=str(tmp_path / "libscalesim_sanitized.so"), sanitize=True)
    env = dict(os.environ, SCALESIM_LIB=lib, LD_PRELOAD=_asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    which = subprocess.run([sys.executable, "-c", "from paper_2601_21473_amd import binding as B; "
                            "print(B.load()._name)"], env=env, cwd=ROOT, capture_output=True,
                           text=True, timeout=120)
    assert which.returncode == 0 and which.stdout.strip() == lib, which.stdout + which.stderr
    # the struct-layout test compiles and runs a C program of its own; the
    # other tests call every entry point's argument checks
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"), "-k", "not struct_layouts"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
