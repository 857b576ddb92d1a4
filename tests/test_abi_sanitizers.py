"""librslm's host-side argument validation under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: the library's sources are compiled
with the sanitizers on their host code only (hipcc ``-Xarch_host``; the device code
is compiled as usual but never launched), linked with tests/abi_sanitize_driver.cpp, and the driver
calls every entry point with arguments that must be rejected before any
launch.  The driver exits non-zero on a wrong status; the sanitizers abort on
any memory or undefined-behaviour error in the host code it reaches."""

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/lib/llvm/bin/clang++"
ROCM_LIB = "/opt/rocm/lib"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("abi_san")
    csrc = os.path.join(ROOT, "paper_2608_30384_amd", "csrc")
    srcs = sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))

    def compile_one(src):
        obj = os.path.join(out, os.path.basename(src)[:-4] + ".o")
        cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC",
               "-Xarch_host", "-g", *SAN,
               "-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 2)) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = os.path.join(out, "abi_sanitize_driver")
    drv = os.path.join(out, "driver.o")
    host = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
            "-fno-omit-frame-pointer"]
    for cmd in ([CLANG, "-O1", "-g", "-std=c++17", *host, "-c",
                 os.path.join(ROOT, "tests", "abi_sanitize_driver.cpp"), "-o", drv],
                [CLANG, *host, drv, *objs, "-L", ROCM_LIB, "-lamdhip64",
                 "-Wl,-rpath," + ROCM_LIB, "-o", exe]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
    yield exe
    shutil.rmtree(out, ignore_errors=True)


def test_validation_paths_are_clean_under_sanitizers(driver):
    env = dict(os.environ)
    # the HIP runtime's own allocations are not this library's: no leak check
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["HIP_VISIBLE_DEVICES"] = ""
    r = subprocess.run([driver], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "ok (0 failures)" in r.stdout
