"""The host runtime (the C ABI's validation, tree metadata, size queries,
argument checks and context creation/teardown) built as plain C++ with
AddressSanitizer and UndefinedBehaviorSanitizer, run on the CPU against the
checks in tests/host_asan/driver.cpp.  The kernels are replaced by stubs
that report an error, so no device work is reached."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang++"


@pytest.mark.skipif(not os.path.exists(CLANG), reason="ROCm clang++ not installed")
def test_host_runtime_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "tss_host_sanitized")
    sanitize = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    cmd = [CLANG, "-std=c++17", "-O1", "-g", "-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2609_26100_amd", "csrc"),
           *sanitize, "-Wno-everything",
           os.path.join(ROOT, "paper_2609_26100_amd", "csrc", "tss_host.cpp"),
           os.path.join(ROOT, "tests", "host_asan", "stub_launchers.cpp"),
           os.path.join(ROOT, "tests", "host_asan", "driver.cpp"),
           "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    # no GPU visible to the check: creation must fail in its HIP set-up and clean up
    env["HIP_VISIBLE_DEVICES"] = ""
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "host sanitizer checks passed" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
