"""AddressSanitizer + UndefinedBehaviorSanitizer build of the library's host code (CPU only).

The C-ABI layer (argument validation, workspace layout, launch set-up in every
.hip source's host pass) and the scheduling simulation are compiled with both
sanitizers, linked with `tests/native/sanitize_host.cpp`, and run. The driver
only makes calls that fail validation, run host code, or (without a GPU)
reach the HIP runtime and must return RP_ERR_HIP; any sanitizer report or
failed expectation fails the test. Device code is built as usual: the
sanitizer flags apply to the host pass only.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2606_26997_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))
DRIVER = os.path.join(HERE, "native", "sanitize_host.cpp")
CLANG = "/opt/rocm/llvm/bin/clang++"

# Host-pass sanitizer flags for hipcc: each one behind -Xarch_host so that
# the device pass is untouched.
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
CPP_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    return r.returncode, r.stdout


@pytest.fixture(scope="module")
def sanitized_exe(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("ROCm clang++ not found")
    out = tmp_path_factory.mktemp("san")
    hipcc = B.hipcc()
    flags = [f for f in B.HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"]

    def hip_obj(src):
        obj = str(out / (src + ".o"))
        rc, log = _run([hipcc, *flags, *HOST_SAN, "-c", os.path.join(B.CSRC, src), "-o", obj])
        assert rc == 0, log
        return obj

    def cpp_obj(path):
        obj = str(out / (os.path.basename(path) + ".o"))
        rc, log = _run([CLANG, "-O1", "-g", "-std=c++17", "-fPIC", "-ffp-contract=off", *CPP_SAN,
                        "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", B.INCLUDE, "-I", B.CSRC,
                        "-c", path, "-o", obj])
        assert rc == 0, log
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(hip_obj, B.SOURCES))
        objs += list(ex.map(cpp_obj, [os.path.join(B.CSRC, s) for s in B.HOST_SOURCES] + [DRIVER]))
    exe = str(out / "sanitize_host")
    rc, log = _run([hipcc, f"--offload-arch={B.ARCH}", "-fsanitize=address", "-fsanitize=undefined",
                    "-fno-gpu-sanitize", *objs, "-o", exe])
    assert rc == 0, log
    return exe


def test_host_code_under_asan_and_ubsan(sanitized_exe):
    env = dict(os.environ)
    # The HIP runtime keeps some allocations until exit; leaks are not what this run checks.
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    rc, log = _run([sanitized_exe], env=env, timeout=300)
    assert rc == 0, log
    assert "all expectations held" in log, log
    assert "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log
