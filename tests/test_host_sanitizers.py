"""Host-side AddressSanitizer + UndefinedBehaviorSanitizer run of the C ABI
layer: every library source compiled with both sanitizers on its host side
only (the gfx950 device code is built as usual and never launched), linked
with the driver tests/sanitize/abi_driver.cpp, which
exercises every argument check, the workspace planning over many shapes,
the canonical converters and the status, debug and timing calls.  The run
must report no sanitizer finding and no failed expectation.  CPU only."""
import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANGXX = "/opt/rocm/llvm/bin/clang++"

pytestmark = [pytest.mark.skipif(not os.path.exists(HIPCC), reason="ROCm toolchain absent"), pytest.mark.slow]


def test_abi_under_asan_and_ubsan(tmp_path):
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined"]
    common = ["-O1", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include")]
    dev = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        r = subprocess.run([HIPCC, *dev, *common, *san, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2605_03667_amd", "csrc", "*.hip")))
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    # the driver is plain C++ (host only), compiled on its own line
    drv = os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp")
    drv_obj, exe = str(tmp_path / "abi_driver.o"), str(tmp_path / "abi_driver")
    r = subprocess.run([CLANGXX, *common, "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-c", drv,
                        "-o", drv_obj], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([HIPCC, *dev, *san, drv_obj, *objs, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                        "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1",
               HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "abi driver: 0 failures" in out
