"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The C oracle with a driver (tests/sanitize/oracle_check.c) that runs it on
  400 seeded random DAGs, the degenerate graphs and every documented error,
  checking the definitions it claims along the way.
* The C ABI's host code: every source of the library built with the
  sanitizers on its host side only (device code is built as usual and never
  runs here), linked with a driver (tests/sanitize/abi_host_check.c) that
  calls every entry point on the paths a machine without a GPU reaches:
  argument checks, NULL handles, status and error text, the
  allocation-failure hook and E_DEVICE.
A sanitizer finding aborts the driver, so each test asserts a clean exit.
"""
import glob
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
SAN_ENV.pop("PARDNN_FAULT_ALLOC", None)


def run_clean(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=SAN_ENV, timeout=300)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report
    assert "all passed" in r.stdout, report
    assert "runtime error" not in report and "Sanitizer" not in report, report


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_check")
    subprocess.run(["gcc", "-std=c99", "-O1", "-g", "-Wall", "-Werror",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "oracle"),
                    os.path.join(ROOT, "oracle", "pardnn_oracle.c"),
                    os.path.join(HERE, "oracle_check.c"), "-o", exe], check=True)
    run_clean(exe)


HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/lib/llvm/bin/clang"


@pytest.mark.skipif(not os.path.exists(HIPCC) or not os.path.exists(CLANG),
                    reason="needs the ROCm toolchain")
@pytest.mark.skipif(torch.cuda.is_available(),
                    reason="checks the paths of a machine without a GPU")
def test_abi_host_code_under_asan_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2008_08636_amd", "csrc")
    inc = os.path.join(ROOT, "include")
    # the sanitizers instrument the host side only: each -fsanitize option
    # follows -Xarch_host
    host_san = ["-Xarch_host", "-fsanitize=address,undefined",
                "-Xarch_host", "-fno-sanitize-recover=all",
                "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        *host_san, "-I", inc, "-I", csrc, "-c", src, "-o", obj],
                       check=True, capture_output=True)
        return obj

    srcs = sorted(glob.glob(os.path.join(csrc, "*.hip")))
    with ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(compile_one, srcs))
    drv = str(tmp_path / "abi_host_check.o")
    subprocess.run([CLANG, "-std=c99", "-O1", "-g", "-Wall", "-Werror",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I", inc,
                    "-c", os.path.join(HERE, "abi_host_check.c"), "-o", drv], check=True)
    exe = str(tmp_path / "abi_host_check")
    subprocess.run([CLANG + "++", "-fsanitize=address,undefined", "-o", exe, *objs, drv,
                    "-L/opt/rocm/lib", "-lamdhip64", "-lrocprofiler-sdk-roctx",
                    "-Wl,-rpath,/opt/rocm/lib"], check=True)
    run_clean(exe)
