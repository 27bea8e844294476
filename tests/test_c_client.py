"""The C ABI from a plain C11 program (tests/c_client/abi_client.c): the
header compiles as C, the library links without Python or torch, and the
calls behave as include/boxconv.h states."""
import os
import shutil
import subprocess

import pytest

from paper_1906_11367_amd import boxconv as bc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_client", "abi_client.c")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

pytestmark = pytest.mark.skipif(not os.path.exists(bc.LIB_PATH) or shutil.which("gcc") is None,
                                reason="libboxconv.so not built or no C compiler")


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("c_client") / "abi_client")
    libdir = os.path.dirname(bc.LIB_PATH)
    cmd = ["gcc", "-std=c11", "-Wall", "-Werror", "-Wno-unused-function", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-L", libdir, "-lboxconv", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           f"-Wl,-rpath,{libdir}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def test_c_client_argument_checks(client):
    r = subprocess.run([client, "check"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


@pytest.mark.gpu
def test_c_client_fwd_bwd_on_gpu(client):
    r = subprocess.run([client, "run"], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
