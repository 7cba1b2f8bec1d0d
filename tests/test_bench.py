"""bench.py on the CPU: its byte model per parameter (the table of
algorithmic bytes each kernel moves), the single-GPU refusal, and the rule
that counter traffic from a committed profile is used only while the kernel
source it was measured on is unchanged."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("algo,g_bytes,deferred,want", [
    # LAMB: read x g m v, write m v; then read x m v, write x
    ("lamb", 2, False, (22, 16)),
    ("lamb", 4, False, (24, 16)),
    # N-LAMB / NN-LAMB read g again in the apply pass
    ("nlamb", 2, False, (22, 18)),
    ("nnlamb", 4, False, (24, 20)),
    # LARS: read x g m, write m; then read x m, write x
    ("lars", 2, False, (14, 12)),
    ("lars", 4, False, (16, 12)),
    # deferred: the moment pass only reads; the apply pass reads x g m v and
    # writes x m v
    ("lamb", 2, True, (14, 26)),
    ("lars", 2, True, (10, 18)),
])
def test_two_pass_bytes(algo, g_bytes, deferred, want):
    assert bench.bytes_per_param(algo, g_bytes, deferred) == want


@pytest.mark.parametrize("algo,g_bytes,want", [("lamb", 2, 26), ("lamb", 4, 28),
                                               ("nnlamb", 2, 26), ("lars", 2, 18),
                                               ("lars", 4, 20)])
def test_single_pass_bytes_are_the_single_touch_floor(algo, g_bytes, want):
    # x, g and the moments read once; x and the moments written once
    assert bench.single_pass_bytes(algo, g_bytes) == want


def test_stream_patterns_match_the_kernels():
    assert bench.pattern_bytes("single_pass", 2) == bench.single_pass_bytes("lamb", 2)
    assert bench.pattern_bytes("moments", 2) == bench.bytes_per_param("lamb", 2)[0]
    assert bench.pattern_bytes("apply", 2) == bench.bytes_per_param("lamb", 2)[1]
    assert bench.pattern_bytes("copy", 2) == 8


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr
    assert r.stdout.strip() == "" or not r.stdout.strip().startswith("{")


def test_counter_traffic_only_for_the_profiled_kernel(tmp_path, monkeypatch):
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    assert h == bench.kernel_source_hash()  # stable
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.counter_traffic("single_pass", "bert-large", h) is None  # no file
    path = tmp_path / "lamb_single_pass_bert-large_traffic.md"
    path.write_text("kernel_source_hash: %s\nhbm_bytes_per_launch: 7.9e+09\n" % h)
    assert bench.counter_traffic("single_pass", "bert-large", h) == pytest.approx(7.9e9)
    path.write_text("kernel_source_hash: 0123456789abcdef\nhbm_bytes_per_launch: 7.9e+09\n")
    assert bench.counter_traffic("single_pass", "bert-large", h) is None  # stale


def test_source_hash_ignores_comments_and_blank_lines():
    code = "int f(int a) {\n    return a + 1;  // one more\n}\n"
    same = "/* header\n   comment */\n\nint f(int a) {\n    // note\n    return a + 1;\n}\n\n"
    other = "int f(int a) {\n    return a + 2;\n}\n"
    assert bench._strip_comments(code) == bench._strip_comments(same)
    assert bench._strip_comments(code) != bench._strip_comments(other)
