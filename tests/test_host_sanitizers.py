"""The library's host code (scheduler, allocator, coordinator decisions, C ABI) under
AddressSanitizer and UndefinedBehaviorSanitizer: a build of libhxf.so with only the
host code instrumented runs the CPU parity suites of the scheduler, the workflow
driver and the coordinator in a child process.  Device code is not instrumented and
no GPU is used."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2505_05286_amd")
# instrumentation applies to the host compilation only
HOST_FLAGS = ["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]
LINK_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"]
SUITES = ["tests/test_sched_parity.py", "tests/test_workflows.py", "tests/test_cluster_parity.py",
          "tests/test_decode_plan.py", "tests/test_abi.py"]


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.slow
def test_host_code_under_address_and_ub_sanitizers():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime in this toolchain")
    from paper_2505_05286_amd import build
    out = os.path.join(PKG, "_build_san", "libhxf_san.so")
    build.build(out=out, build_dir=os.path.dirname(out), host_flags=HOST_FLAGS, link_flags=LINK_FLAGS)
    env = dict(os.environ, LD_PRELOAD=rt, HXF_LIBRARY=out,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu and not slow",
                        "-p", "no:cacheprovider"] + SUITES, cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=1200)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
