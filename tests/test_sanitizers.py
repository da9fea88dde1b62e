"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The library's synchronous host helpers (api.cpp: topology table, path
validation, draft pruning and packing, the tree-mask converter, the
argument checks) and the C oracle are compiled with g++/gcc and
-fsanitize=address,undefined (no GPU code: the kernel launchers are stubbed
in the driver) and driven by tests/sanitize_driver.cpp over exhaustive small
drafts, random drafts up to the size limits and malformed inputs.  Any
out-of-bounds access, use after free, leak or undefined behaviour aborts the
run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_16673_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
# the sanitizer runtimes linked statically: they need not come first among
# the process's shared libraries, so the environment is used as it is
LINK = ["-static-libasan", "-static-libubsan"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc/g++")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    hip_inc = "/opt/rocm/include"
    if not os.path.exists(os.path.join(hip_inc, "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not installed")
    objs = []
    cxx = ["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           "-I" + hip_inc, "-Wno-deprecated-declarations"] + SAN
    for name, src in [("api", os.path.join(CSRC, "api.cpp")),
                      ("driver", os.path.join(ROOT, "tests", "sanitize_driver.cpp"))]:
        obj = str(tmp_path / (name + ".o"))
        r = subprocess.run(cxx + ["-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        objs.append(obj)
    obj = str(tmp_path / "oracle.o")
    r = subprocess.run(["gcc", "-std=c11", "-ffp-contract=off", "-c", os.path.join(ROOT, "oracle", "oracle.c"),
                        "-o", obj] + SAN, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    objs.append(obj)
    exe = str(tmp_path / "sanitize_driver")
    r = subprocess.run(["g++"] + SAN + LINK + objs + ["-lm", "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-6000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-6000:]
    assert "sanitized host checks passed" in out
