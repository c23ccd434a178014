"""The host side of the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

api.cpp, validate.cpp and plan.cpp -- every argument check, status and plan
the entry points compute before launching anything -- are built with g++
-fsanitize=address,undefined into a library whose kernel launchers are
test stand-ins (tests/hostsan/launch_stubs.cpp), and every case of
tests/test_abi.py runs against it in a child process with the ASan runtime
preloaded; any sanitizer report fails the run."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_18502_amd", "csrc")
ROCM_INCLUDE = "/opt/rocm/include"


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if shutil.which("g++") is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("g++ or the HIP headers are not available")
    if _runtime("libasan.so") is None:
        pytest.skip("no AddressSanitizer runtime")
    out = str(tmp_path_factory.mktemp("hostsan") / "libspecfp8_hostsan.so")
    srcs = [os.path.join(CSRC, f) for f in ("api.cpp", "validate.cpp", "plan.cpp")]
    srcs.append(os.path.join(ROOT, "tests", "hostsan", "launch_stubs.cpp"))
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__",
           f"-I{ROCM_INCLUDE}", f"-I{os.path.join(ROOT, 'include')}", *srcs, "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return out


def test_abi_cases_under_sanitizers(sanitized_lib):
    env = dict(os.environ)
    env["LD_PRELOAD"] = _runtime("libasan.so")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["SPECFP8_ABI_LIB"] = sanitized_lib
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=300)
    log = res.stdout + res.stderr
    assert res.returncode == 0, log[-4000:]
    assert "ERROR: AddressSanitizer" not in log and "runtime error:" not in log, log[-4000:]
    assert " passed" in log
