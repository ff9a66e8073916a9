"""The C ABI's host code under AddressSanitizer, without a GPU.

The library's host-side sources (argument checks, buffer carving, size
queries, the trace API, the static-scratch lookup) are rebuilt with
AddressSanitizer on the host pass only, linked with the kernels' objects of
the regular build, and driven by a C program (`abi_asan_driver.c`) through
every size query, view query and argument-error path of every entry point,
the trace API and the per-thread error strings.  A heap or stack overflow, a
use after free or a leak in that code fails the run."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_00916_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"
# instrumented: the sources whose host code does more than launch kernels
HOST_SOURCES = ("moe_api.cpp", "trace.cpp", "noalloc.hip")
# host pass only: the device code is built as in the library
ASAN_HOST = "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer".split()


def kernel_objects():
    names = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")) and f not in HOST_SOURCES)
    return [os.path.join(BUILD, n + ".o") for n in names]


def run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not installed")
def test_abi_host_code_under_asan(tmp_path):
    objs = kernel_objects()
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        pytest.skip(f"kernel objects of the regular build missing (build first): {missing}")
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Wno-unused-function",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC, *ASAN_HOST]
    procs = []
    host_objs = []
    for src in HOST_SOURCES:
        o = str(tmp_path / (src + ".o"))
        host_objs.append(o)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", o],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
    for p in procs:
        out, err = p.communicate()
        assert p.returncode == 0, err
    lib = str(tmp_path / "libmoe_asan.so")
    run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", lib, *host_objs, *objs])
    exe = str(tmp_path / "abi_driver")
    run([CLANG, "-std=c99", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
         "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "abi_asan_driver.c"),
         f"-L{tmp_path}", "-lmoe_asan", f"-Wl,-rpath,{tmp_path}", "-lpthread", "-lm", "-o", exe])
    args = [exe] if os.path.exists("/dev/kfd") else [exe, "launch"]  # no GPU: a refused launch too
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1")
    r = subprocess.run(args, capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, f"{r.stdout}\n{r.stderr}"
    assert "0 failure(s)" in r.stdout
    assert "AddressSanitizer" not in r.stderr and "LeakSanitizer" not in r.stderr, r.stderr
