"""Host C++ of libtsr under AddressSanitizer and UndefinedBehaviorSanitizer.

The planner, the C ABI's validation, the context-unit cache directory and
the control plane (the .cpp sources) are compiled with g++ and
-fsanitize=address,undefined and linked with the GPU kernels' objects of
the normal build into a separate library; the host-only test modules then
run against it (TSR_LIBRARY) in a child process with the sanitizer runtimes
preloaded.  Any report fails the test.  CPU only: no kernel is launched.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32999_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
OUT = os.path.join(BUILD, "asan")
MODULES = ["tests/test_abi.py", "tests/test_unit_cache.py", "tests/test_control_plane.py"]
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]


def _gxx_runtime(name):
    return subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True,
                          text=True, check=True).stdout.strip()


def _build_sanitized() -> str:
    """Host sources with sanitizers (g++), kernel objects as normally built."""
    from paper_2609_32999_amd.build_lib import build
    kernel_objs = sorted(glob.glob(os.path.join(BUILD, "*.hip.o")))
    if not kernel_objs:
        build()
        kernel_objs = sorted(glob.glob(os.path.join(BUILD, "*.hip.o")))
    os.makedirs(OUT, exist_ok=True)
    host_objs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.cpp"))):
        obj = os.path.join(OUT, os.path.basename(src) + ".o")
        cmd = ["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
               "-I" + os.path.join(ROOT, "include"), *SAN, "-g", "-O1", "-fPIC",
               "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        host_objs.append(obj)
    lib = os.path.join(OUT, "libtsr_asan.so")
    cmd = ["g++", "-shared", *SAN, "-o", lib, *host_objs, *kernel_objs, "-L/opt/rocm/lib",
           "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return lib


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime.h"),
                    reason="ROCm headers are needed to build the host sources")
def test_host_code_is_clean_under_asan_and_ubsan():
    lib = _build_sanitized()
    env = dict(os.environ)
    env.update({
        "TSR_LIBRARY": lib,
        "LD_PRELOAD": _gxx_runtime("libasan.so") + ":" + _gxx_runtime("libubsan.so"),
        # the interpreter itself is not instrumented: its allocations are not
        # leaks of ours; every other report aborts the child
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    probe = ("import paper_2609_32999_amd._binding as B; B.lib(); "
             "maps = open('/proc/self/maps').read(); "
             "assert 'libtsr_asan.so' in maps and 'libasan' in maps, 'not sanitized'; "
             "print('sanitized library loaded:', B.LIB_PATH)")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *MODULES], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
