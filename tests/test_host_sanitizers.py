"""The library's host C++ under AddressSanitizer and UndefinedBehaviorSanitizer.

abi.cpp holds the host logic of the boundary: the arena and its free list, the
stash layout of Eq. 12, shard validation and the memory estimate of Sec. 3 and
Sec. 4.1.  This test rebuilds it with host-side sanitizers (device code is
unchanged), links it with the kernel objects of the regular build, and runs the
host tests of test_abi_host.py against that library in a child process with
the sanitizer runtime preloaded.  Undefined behaviour aborts the child, so any
report fails the test.  No GPU is touched.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2411_06465_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# host-side only: each sanitizer flag applies to the host compilation
HOST_SAN = "-Xarch_host -fsanitize=address,undefined -Xarch_host -fno-sanitize-recover=undefined".split()
HOST_FP = "-Xarch_host -fno-omit-frame-pointer".split()
KERNEL_SOURCES = ["gemm.hip", "attention.hip", "rowwise.hip", "optim.hip"]


def _asan_runtime():
    found = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed:\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    runtime = _asan_runtime()
    if not os.path.exists(HIPCC) or runtime is None:
        pytest.skip("hipcc or the clang AddressSanitizer runtime is not installed")
    sys.path.insert(0, ROOT)
    from paper_2411_06465_amd import build as B

    objs = []
    for src in KERNEL_SOURCES:      # the regular build's objects when present, else compiled here
        obj = os.path.join(PKG, "_build", os.path.splitext(src)[0] + ".o")
        objs.append(obj if os.path.exists(obj) else B._compile(src, str(tmp_path)))
    flags = [f for f in B.FLAGS if f != "-O3"] + ["-O1", "-g"]
    abi = str(tmp_path / "abi_san.o")
    _run([HIPCC, *flags, *HOST_SAN, *HOST_FP, "-c", os.path.join(PKG, "csrc", "abi.cpp"), "-o", abi])
    lib = str(tmp_path / "libl4d_san.so")
    _run([HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *HOST_SAN, "-shared-libsan", "-o", lib, abi, *objs])

    env = dict(os.environ, L4D_LIB=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0",          # the interpreter's own allocations are not ours
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"), "-q",
                        "-p", "no:cacheprovider"], capture_output=True, text=True, env=env, cwd=ROOT)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0 and " passed" in out, out[-4000:]
