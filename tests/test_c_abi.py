"""The C ABI from C: both public headers compile as C99 and C++11 with
warnings as errors, and a plain C program (tests/c_abi_consumer.c) linked
against the library gets the documented results from every host-only entry
point (status strings, defaults, chunk table, tile schedule, learning-rate
schedule, argument validation). Nothing here touches a GPU."""

import os
import shutil
import subprocess

import pytest

from paper_1904_00962_amd import build

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(build.LIBRARY)


def _compiler(name):
    path = shutil.which(name)
    if path is None:
        pytest.skip("%s is not installed" % name)
    return path


@pytest.mark.parametrize("lang,std", [("c", "-std=c99"), ("c++", "-std=c++11")])
def test_headers_compile_standalone(tmp_path, lang, std):
    cc = _compiler("gcc" if lang == "c" else "g++")
    src = tmp_path / ("h.c" if lang == "c" else "h.cpp")
    src.write_text('#include "lamb_mi355x.h"\n#include "stream_probe.h"\n'
                   "int main(void) { return (int)LAMB_OK; }\n")
    r = subprocess.run([cc, std, "-Wall", "-Wextra", "-Werror", "-pedantic", "-fsyntax-only",
                        "-I", build.INCLUDE, str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_program_uses_the_host_entry_points(tmp_path):
    cc = _compiler("gcc")
    if build.is_stale():
        build.build()
    exe = tmp_path / "consumer"
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                        "-I", build.INCLUDE, os.path.join(HERE, "c_abi_consumer.c"),
                        "-L", PKG, "-l:" + os.path.basename(build.LIBRARY),
                        "-Wl,-rpath," + PKG, "-lm", "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


def test_host_code_under_sanitizers(tmp_path):
    """The library's host code (lamb_api.cpp: validation, chunk table, tile
    schedule, learning-rate helpers, status strings) built with g++ under
    AddressSanitizer and UndefinedBehaviorSanitizer, with the kernel
    launchers stubbed (tests/host_only_stubs.cpp), and driven by the same C
    program: any out-of-bounds access, leak or undefined behaviour (such as
    an out-of-range enum value) fails the run."""
    gxx, gcc = _compiler("g++"), _compiler("gcc")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    if not os.path.exists(os.path.join(rocm, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not found under %s" % rocm)
    san = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    lib = tmp_path / "liblamb_host_san.so"
    r = subprocess.run([gxx, "-std=c++17", "-O1", "-g", *san, "-fPIC", "-shared",
                        "-D__HIP_PLATFORM_AMD__", "-I", build.INCLUDE, "-I", build.CSRC,
                        "-I", os.path.join(rocm, "include"),
                        os.path.join(build.CSRC, "lamb_api.cpp"),
                        os.path.join(HERE, "host_only_stubs.cpp"),
                        "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                        "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", str(lib)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    exe = tmp_path / "consumer_san"
    r = subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", *san,
                        "-I", build.INCLUDE, os.path.join(HERE, "c_abi_consumer.c"),
                        "-L", str(tmp_path), "-l:" + lib.name, "-Wl,-rpath," + str(tmp_path),
                        "-lm", "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout and "runtime error" not in r.stderr
