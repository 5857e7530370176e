"""The C ABI from a plain C program on the GPU (tests/native/abi_gpu_c.c): HIP runtime buffers,
tvq_create, tvq_encode and tvq_decode with no Python binding in between; the program checks
the cache against the oracle's encode (codes outside the flag zone, headers within 2 ulp) and
the fp32 decode against the oracle's fp64 decode of the GPU's cache."""
import os
import shutil
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_program_encodes_and_decodes_through_the_abi(gpu, tmp_path):
    import paper_2603_27467_amd as tvq
    import oracle
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("gcc not found")
    lib = tvq.library_path()
    olib = oracle.library_path()
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    exe = str(tmp_path / "abi_gpu_c")
    subprocess.run([cc, "-std=c99", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
                    "-I", os.path.join(rocm, "include"),
                    os.path.join(ROOT, "tests", "native", "abi_gpu_c.c"), lib, olib,
                    "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-lm",
                    "-Wl,-rpath," + ":".join([os.path.dirname(lib), os.path.dirname(olib),
                                              os.path.join(rocm, "lib")]),
                    "-o", exe], check=True)
    print("running the C program", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    sys.stdout.write(r.stdout)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
