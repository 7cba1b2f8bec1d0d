"""The optimizer step from a plain C program (tests/c_gpu_consumer.c): device
buffers from the HIP runtime, LAMB on both paths with fp32 and bf16
gradients and LARS through include/lamb_mi355x.h, each step checked against
the C oracle library on the same inputs, with the tolerances of the Python
parity harness. The boundary needs neither Python nor torch."""

import os
import shutil
import subprocess

import pytest

import gpu_harness as H
from paper_1904_00962_amd import build

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ORACLE_DIR = os.path.join(ROOT, "oracle")


def test_c_program_steps_on_the_gpu(tmp_path):
    H.torch_cuda()
    gcc = shutil.which("gcc")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    if gcc is None or not os.path.exists(os.path.join(rocm, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("gcc or the HIP headers are missing")
    oracle_lib = os.path.join(ORACLE_DIR, "liblamb_oracle.so")
    assert os.path.exists(build.LIBRARY) and os.path.exists(oracle_lib), "run the build first"
    pkg = os.path.dirname(build.LIBRARY)
    exe = tmp_path / "c_gpu_consumer"
    r = subprocess.run([gcc, "-std=c99", "-O1", "-Wall", "-Wextra", "-Werror",
                        "-D__HIP_PLATFORM_AMD__", "-I", build.INCLUDE,
                        "-I", os.path.join(rocm, "include"),
                        os.path.join(HERE, "c_gpu_consumer.c"),
                        "-L", pkg, "-l:" + os.path.basename(build.LIBRARY),
                        "-L", ORACLE_DIR, "-l:liblamb_oracle.so",
                        "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                        "-Wl,-rpath," + ":".join([pkg, ORACLE_DIR, os.path.join(rocm, "lib")]),
                        "-lm", "-o", str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    H.log("c consumer: LAMB fp32/bf16 on both paths and LARS, 3 steps each, 7 ragged tensors")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(r.stdout, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
