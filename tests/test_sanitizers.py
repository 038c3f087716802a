"""The CPU oracle and the C ABI's host code under sanitizers (no GPU needed).

* The oracle (oracle/dart_oracle.c) is built with gcc under AddressSanitizer
  and UndefinedBehaviorSanitizer, with and without OpenMP, and
  tests/sanitize/oracle_driver.c runs every oracle function on small shapes
  with exactly sized buffers.
* The ABI's host side (dart_api.cpp, profile.cpp) is built with the host half
  of hipcc under ASan + UBSan and, separately, ThreadSanitizer, and linked with
  the library's other objects; tests/sanitize/abi_driver.c runs the workspace
  sizing and argument-rejection paths and calls the profiling functions from
  four threads.
Any sanitizer report aborts the driver (-fno-sanitize-recover) and fails the
test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
BUILD = os.path.join(ROOT, "_build")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", OMP_NUM_THREADS="4")


def run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, env=ENV, timeout=600, **kw)
    assert res.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), res.stdout[-3000:], res.stderr[-6000:])
    return res.stdout


@pytest.mark.parametrize("openmp", [False, True])
def test_oracle_under_asan_ubsan(tmp_path, openmp):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_driver")
    cmd = ["gcc", "-O1", "-g", "-std=c99", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-o", exe, os.path.join(SAN, "oracle_driver.c"),
           os.path.join(ROOT, "oracle", "dart_oracle.c"), "-lm"]
    if openmp:
        cmd.insert(1, "-fopenmp")
    run(cmd)
    assert "oracle driver ok" in run([exe])


def library_objects():
    if not os.path.isdir(BUILD):
        return None
    objs = [os.path.join(BUILD, f) for f in sorted(os.listdir(BUILD))
            if f.endswith(".o") and f not in ("dart_api.o", "profile.o")]
    return objs or None


@pytest.mark.parametrize("sanitizers,args", [(["address", "undefined"], []), (["thread"], ["threads"])])
def test_abi_host_code_under_sanitizers(tmp_path, sanitizers, args):
    objs = library_objects()
    if objs is None or not os.path.exists(HIPCC) or not os.path.exists(CLANG):
        pytest.skip("needs hipcc, the ROCm clang and the library objects of a build")
    host = []
    for s in sanitizers:  # host half only: device code is never instrumented
        host += ["-Xarch_host", "-fsanitize=" + s]
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2608_02032_amd", "csrc")]
    mine = []
    for src in ("dart_api.cpp", "profile.cpp"):
        o = str(tmp_path / (src + ".o"))
        run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature",
             "-Xclang", "-packed-fp32-ops", "-fno-omit-frame-pointer", "-x", "hip"] + host + inc +
            ["-c", os.path.join(ROOT, "paper_2608_02032_amd", "csrc", src), "-o", o])
        mine.append(o)
    drv = str(tmp_path / "abi_driver.o")
    run([CLANG, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=" + ",".join(sanitizers),
         "-fno-sanitize-recover=all", "-I" + os.path.join(ROOT, "include"), "-c",
         os.path.join(SAN, "abi_driver.c"), "-o", drv])
    exe = str(tmp_path / "abi_driver")
    run([HIPCC, "--offload-arch=gfx950"] + host + ["-o", exe, drv] + mine + objs + ["-lpthread"])
    assert "abi driver ok" in run([exe] + args)
