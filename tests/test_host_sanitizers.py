"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

bc_api.cpp (argument checks, workspace arithmetic, path choice, launch
set-up) and bc_noalloc.hip (the fixed-array entry point) are rebuilt with the
sanitizers on their host pass only (each -fsanitize= behind -Xarch_host: the
device code is built as usual), linked with the kernel objects of the normal
build, and the plain C client of tests/c_client runs its argument-check mode
against that library: every rejected size, dtype, alignment, flag and
workspace request goes through the sanitized code, and any overflow, invalid
enum load, out-of-bounds access or other undefined behaviour ends the run.
No GPU is used: every call of the check mode is rejected, or answered, before
a launch.
"""
import os
import shutil
import subprocess

import pytest

from paper_1906_11367_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
SANITIZED = ["bc_api.cpp", "bc_noalloc.hip"]
KERNELS = [s for s in B.SOURCES if s not in SANITIZED]

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                                reason="no hipcc")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-3000:] + r.stderr[-3000:]
    return r


@pytest.fixture(scope="module")
def sanitized_client(tmp_path_factory):
    d = tmp_path_factory.mktemp("sanitized")
    kernel_objs = [os.path.join(B.BUILD, s + ".o") for s in KERNELS]
    if not all(os.path.exists(o) for o in kernel_objs):
        B.build()
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in B.common_flags() if f != "-O3"] + ["-O1", "-g"] + host_san
    objs = []
    for s in SANITIZED:
        o = str(d / (s + ".o"))
        _run([B.hipcc(), *flags, "-x", "hip", "-c", os.path.join(B.CSRC, s), "-o", o])
        objs.append(o)
    lib = str(d / "libboxconv.so")
    _run([B.hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, *kernel_objs, "-o", lib])
    exe = str(d / "abi_client")
    _run([CLANG, "-std=c11", "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
          os.path.join(ROOT, "tests", "c_client", "abi_client.c"), "-L", str(d), "-lboxconv",
          "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm", f"-Wl,-rpath,{d}",
          f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe])
    return exe


def test_argument_checks_clean_under_asan_and_ubsan(sanitized_client):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sanitized_client, "check"], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-3000:] + r.stderr[-3000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-3000:]
