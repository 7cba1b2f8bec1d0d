"""The kernels' resource use, read from the gfx950 assembly hipcc writes for
lamb_kernels.hip and lamb_static.hip (on the CPU; no GPU involved): no kernel spills to scratch,
and every single-pass variant fits the four workgroups per CU that its
persistent grid needs resident (at most 128 VGPRs at four waves per SIMD, and
LDS for four workgroups within the CU's 160 KB)."""

import os
import re
import subprocess

import pytest

from paper_1904_00962_amd import build

KERNEL_SOURCES = [os.path.join(build.CSRC, name)
                  for name in ("lamb_kernels.hip", "lamb_static.hip")]
LDS_PER_CU = 160 * 1024


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    flags = [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    text = ""
    for src in KERNEL_SOURCES:
        out = tmp_path_factory.mktemp("isa") / (os.path.basename(src) + ".s")
        r = subprocess.run([build.hipcc(), *flags, "-I", build.INCLUDE, "-I", build.CSRC,
                            "--cuda-device-only", "-S", src, "-o", str(out)],
                           capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-2000:]
        text += out.read_text()
    found = {}
    for m in re.finditer(r"^\s*\.amdhsa_kernel\s+(\S+)\s*$(.*?)^\s*\.end_amdhsa_kernel",
                         text, re.M | re.S):
        body = m.group(2)

        def field(name, body=body):
            return int(re.search(r"\.amdhsa_%s\s+(\d+)" % name, body).group(1))

        found[m.group(1)] = {"vgpr": field("next_free_vgpr"),
                             "scratch": field("private_segment_fixed_size"),
                             "lds": field("group_segment_fixed_size")}
    return found


def test_every_kernel_variant_was_found(kernels):
    names = list(kernels)
    # 4 algorithms x 2 gradient dtypes x 3 norms, in both tile shapes
    assert sum("fused_kernel" in n for n in names) == 48
    # 4 algorithms x 2 gradient dtypes x (direct, deferred) x 3 norms
    assert sum("moments_kernel" in n for n in names) == 48
    # 4 algorithms x 2 gradient dtypes x (deferred, direct, direct with the
    # u re-sum in 3 norms)
    assert sum("apply_kernel" in n for n in names) == 40
    for kind in ("segment_kernel", "finalize_kernel", "totals_kernel", "scale_kernel"):
        assert sum(kind in n for n in names) == 3, kind
    assert sum("finite_kernel" in n for n in names) == 2
    assert sum("table_kernel" in n for n in names) == 1


def test_no_kernel_spills(kernels):
    spilled = {n: k["scratch"] for n, k in kernels.items() if k["scratch"]}
    assert not spilled, spilled


def test_single_pass_fits_four_workgroups_per_cu(kernels):
    for name, k in kernels.items():
        if "fused_kernel" not in name:
            continue
        assert k["vgpr"] <= 128, (name, k)
        assert 4 * k["lds"] <= LDS_PER_CU, (name, k)
