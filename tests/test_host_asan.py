"""AddressSanitizer over the library's host code (CPU only): api.hip (argument
validation, aliasing and range checks, dispatch) is rebuilt with the host half
instrumented, linked with the other objects of the regular build, and
tests/test_abi.py runs against that library in a child process with the ASan
runtime preloaded.  Any out-of-bounds access or use-after-free in the host
entry points aborts the child.  Device code is not instrumented."""
from __future__ import annotations

import os
import shlex
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "_build")
OUT = os.path.join(BUILD, "asan")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
RUNTIME = "/opt/rocm/lib/llvm/lib/clang/22/lib/linux/libclang_rt.asan-x86_64.so"
# host-side instrumentation only (each sanitizer flag right after -Xarch_host)
HOST_ASAN = "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer"


def _have_toolchain():
    return os.path.exists(HIPCC) and os.path.exists(RUNTIME)


@pytest.mark.skipif(not _have_toolchain(), reason="hipcc or the clang ASan runtime is missing")
@pytest.mark.timeout(900)
def test_abi_under_host_asan():
    sys.path.insert(0, ROOT)
    from paper_2607_14952_amd import build as b
    objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in b.SOURCES]
    if not all(os.path.exists(o) for o in objs):
        b.build()
    os.makedirs(OUT, exist_ok=True)
    api_obj = os.path.join(OUT, "api.o")
    flags = [f"--offload-arch={b.ARCH}", "-O1", "-g", "-std=c++17", "-fPIC",
             "-fvisibility=hidden", "-I", os.path.join(ROOT, "include"),
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    subprocess.run([HIPCC, *flags, *shlex.split(HOST_ASAN), "-c",
                    os.path.join(b.CSRC, "api.hip"), "-o", api_obj],
                   check=True, capture_output=True)
    lib = os.path.join(OUT, "liblongstraw.so")
    others = [o for o in objs if not o.endswith("api.o")]
    subprocess.run([HIPCC, f"--offload-arch={b.ARCH}", "-shared", "-fPIC",
                    *shlex.split(HOST_ASAN), api_obj, *others, "-o", lib],
                   check=True, capture_output=True)
    env = dict(os.environ, LONGSTRAW_LIB=lib, LD_PRELOAD=RUNTIME,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr, tail
    assert " passed" in r.stdout, tail
