"""AddressSanitizer + UndefinedBehaviorSanitizer build of the library's host code (CPU only).

Every HIP source is compiled with the sanitizers on its host code only (each -fsanitize is
given to the host compiler; the gfx950 device code is built as usual) and linked with
tests/host_sanitize.cpp, a driver that runs the host-side validation paths, workspace
queries, the loss call's slab planner on hundreds of random length mixes, and the adaptive
rollout sampling controller.  Any out-of-bounds access, use after free, signed overflow or
other undefined behaviour in that host code ends the run with a sanitizer report."""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36932_amd", "csrc")
SOURCES = ["api.hip", "advantage.hip", "prune.hip", "lmhead.hip", "optim.hip"]
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
FLAGS = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("host_san")

    def comp(src):
        obj = str(out / (os.path.basename(src) + ".o"))
        r = subprocess.run([hipcc, *FLAGS, *HOST_SAN, "-c", src, "-o", obj],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        return obj

    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    with ThreadPoolExecutor(max_workers=5) as ex:
        objs = list(ex.map(comp, srcs))
    drv = str(out / "host_sanitize.o")
    r = subprocess.run([hipcc, "-O1", "-g", "-std=c++17", *HOST_SAN, "-x", "c++",
                        os.path.join(ROOT, "tests", "host_sanitize.cpp"), "-c", "-o", drv],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    exe = str(out / "host_sanitize")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", *HOST_SAN, drv, *objs, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def test_host_code_under_asan_ubsan(driver):
    env = dict(os.environ)
    # the HIP runtime keeps some allocations until exit; leaks are not what this checks
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([driver], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "HOST_SANITIZE_OK" in r.stdout, (r.stdout[-2000:],
                                                                  r.stderr[-4000:])
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
