"""The library's host C++ (layout.cpp, select.cpp, api.cpp, cnn.cpp,
growth.cpp) built with g++ and AddressSanitizer + UndefinedBehaviorSanitizer
(and LeakSanitizer) against counting HIP stand-ins (tests/host/hip_stub.cpp),
driven by tests/host/host_driver.cpp on the CPU: validation paths, weight
packing, handle lifecycles with an allocation failure at every hipMalloc of
each create, forwards' host-side planning, growth-step argument checks and
the DN selection of Eq. 11.  The driver also counts HIP calls to show that a
DN-mode switch (Section 6.2) makes none and launches nothing, and that a
forward allocates nothing."""
import concurrent.futures as cf
import hashlib
import os
import shutil
import subprocess

import pytest

from paper_2609_10018_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = os.path.join(ROOT, "tests", "host")
OUT = os.path.join(ROOT, "_build", "host_san")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
FLAGS = ["-std=c++17", "-O1", "-g", "-Wall", "-Werror=format", "-D__HIP_PLATFORM_AMD__",
         "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include")] + SAN

pytestmark = pytest.mark.skipif(
    shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include/hip"),
    reason="needs g++ and the HIP headers")


def _sources():
    lib = [os.path.join(build.CSRC, s) for s in build.SOURCES if s.endswith(".cpp")]
    return lib + [os.path.join(HOST, "hip_stub.cpp"), os.path.join(HOST, "host_driver.cpp")]


def _compile(src):
    deps = [src, os.path.join(HOST, "hip_stub.h")] + \
        [os.path.join(build.CSRC, h) for h in os.listdir(build.CSRC) if h.endswith(".h")] + \
        [os.path.join(ROOT, "include", "elasto.h")]
    key = hashlib.sha256(" ".join(FLAGS).encode())
    for d in deps:
        key.update(open(d, "rb").read())
    obj = os.path.join(OUT, f"{os.path.basename(src)}.{key.hexdigest()[:12]}.o")
    if not os.path.exists(obj):
        r = subprocess.run(["g++"] + FLAGS + ["-c", src, "-o", obj + ".tmp"],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        os.replace(obj + ".tmp", obj)
    return obj


@pytest.fixture(scope="module")
def driver():
    os.makedirs(OUT, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, _sources()))
    exe = os.path.join(OUT, "host_driver")
    r = subprocess.run(["g++"] + SAN + ["-o", exe] + objs, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_host_sources_clean_under_asan_ubsan(driver):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([driver], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout[-2000:])
    print(r.stderr[-4000:])
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "0 failed" in r.stdout
    assert "runtime error" not in r.stderr          # UBSan report
    assert "AddressSanitizer" not in r.stderr       # ASan warning or report
    assert "LeakSanitizer" not in r.stderr
