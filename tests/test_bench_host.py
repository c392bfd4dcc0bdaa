"""Host-side logic of bench.py (no GPU): the kernel-source hash that ties
the committed HBM-traffic figures to the kernels they were measured on."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_code_tokens_ignore_comments_and_layout():
    a = "int f(int x) {\n  return x + 1;  // add one\n}\n/* block\n comment */\n"
    b = "int f(int x) { return x + 1; }"
    assert bench._code_tokens(a) == bench._code_tokens(b)


def test_code_tokens_keep_string_and_char_literals():
    src = 'const char* s = "// not a comment /* nor this */"; char c = \'/\'; // gone'
    assert bench._code_tokens(src) == 'const char* s = "// not a comment /* nor this */"; char c = \'/\';'


def test_code_change_changes_tokens():
    assert bench._code_tokens("a = b + 1;") != bench._code_tokens("a = b + 2;")


def test_committed_traffic_figures():
    # profiles/traffic.json holds rocprofv3 counter figures; bench.py reports
    # them only while they were taken on the current kernel code (else null)
    import json
    import pytest
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as fh:
        rec = json.load(fh)
    if rec["kernel_source_hash"] != bench.kernel_source_hash():
        pytest.skip("kernel code changed since the counters were taken")
    assert bench.measured_traffic("gelu_bf16_lm_ffn_16x2048x8192", 3, "fwd") is not None
    for key, v in rec["launches"].items():
        assert 0.99 < v["hbm_bytes"] / v["algorithmic_bytes"] < 1.1, key
