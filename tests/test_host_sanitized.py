"""The library's host code -- descriptor validation, the planner, staging,
timing and the C ABI -- under AddressSanitizer and UndefinedBehaviourSanitizer:
a copy of the library whose host code is sanitized (the GPU kernels are the
regular ones) runs the CPU tests of the ABI (tests/test_abi_host.py) in a child
process with the sanitizer runtime preloaded.  Any report aborts the child.
No GPU is needed: those tests never launch a kernel."""
import os
import subprocess
import sys

from paper_2602_24082_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_host_tests_pass_under_asan_and_ubsan(tmp_path):
    lib = build.build_host_sanitized(str(tmp_path / "libppattn_asan.so"))
    preload = build.asan_runtime()
    if os.environ.get("LD_PRELOAD"):
        preload += ":" + os.environ["LD_PRELOAD"]  # the sanitizer runtime must come first
    env = dict(os.environ, PP_LIB_PATH=lib, LD_PRELOAD=preload,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       env=env, capture_output=True, text=True, cwd=ROOT, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert " passed" in r.stdout and "runtime error" not in out and "AddressSanitizer" not in out, out
