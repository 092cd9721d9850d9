"""Host-side helpers of bench.py that decide whether a stored counter record
still describes the kernels (CPU only)."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_code_only_ignores_comments_and_spacing():
    a = "int x; // note\n/* block\n comment */ int y = 1;\n"
    b = "int x;\n\n    int y = 1;   // another note\n"
    assert bench.code_only(a) == bench.code_only(b) == "int x; int y = 1;"


def test_code_only_keeps_code_changes_and_string_literals():
    assert bench.code_only("int y = 1;") != bench.code_only("int y = 2;")
    # comment markers inside a string literal are code
    assert bench.code_only('const char *s = "a // b"; // c') == 'const char *s = "a // b";'
    assert bench.code_only('s = "q\\"//x"; /* c */') == 's = "q\\"//x";'


def test_source_hash_follows_the_kernel_family():
    gemm = bench.source_hash("gemm_fc1_t256")
    assert gemm == bench.source_hash("gemm_o_t128_ca")
    assert gemm != bench.source_hash("attention_q64_ca")
    assert bench.source_hash("attention_res") == bench.source_hash("attn_scores")
