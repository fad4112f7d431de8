"""CPU checks of bench.py's host-side bookkeeping: the source hash that keys
the committed counter summaries, and the algorithmic byte counts the roofline
divides by."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workload as W  # noqa: E402


def test_code_only_drops_comments_and_layout_but_keeps_strings():
    a = 'int x = 1; // note\n/* block\n comment */ asm("s_nop 0 // not a comment");'
    b = 'int x = 1;\n\n   asm("s_nop 0 // not a comment");   // other note'
    assert bench._code_only(a) == bench._code_only(b)
    assert "// not a comment" in bench._code_only(a)
    assert bench._code_only("int x = 1;") != bench._code_only("int x = 2;")
    assert bench._code_only('"a\\"b" // c') == '"a\\"b"'


def test_committed_counter_summaries_match_the_current_sources():
    """The committed traffic summaries are keyed to the code they were taken
    on; if a kernel's code changes they must be taken again (the bench then
    reports no traffic rather than a stale one)."""
    for kernel, path in (("decode", bench.TRAFFIC_SUMMARY),
                         ("prefill", bench.PREFILL_TRAFFIC_SUMMARY)):
        with open(path) as f:
            t = json.load(f)
        assert t["kernel_src_sha256_16"] == bench.kernel_src_hash(kernel), (
            f"{os.path.basename(path)} was taken on other {kernel} code")
        assert 1.0 <= t["measured_over_algorithmic"] < 1.1


def test_algorithmic_bytes_of_the_headline_workload():
    """Decode: N (|vis| beta + Hq D (b_q + b_o) + 2 beta); prefill: N ((S + W + C - 1)
    beta + C Hq D (b_q + b_o)), plus 2 C beta with the chunk append fused (the
    k, v rows in and the pool copy out), with beta = 2 Hkv D b."""
    dec, pre = bench.algorithmic_bytes(W.QWEN3_OMNI)
    beta = 2 * 4 * 128 * 2
    assert dec == 128 * (4100 * beta + 32 * 128 * 4 + 2 * beta) == 1077411840
    assert pre == 128 * ((4 + 4096 + 25 - 1) * beta + 25 * 32 * 128 * 4)
    _, pre_fused = bench.algorithmic_bytes(W.QWEN3_OMNI, fused_append=True)
    assert pre_fused == pre + 128 * 25 * 2 * beta
    dec8, _ = bench.algorithmic_bytes(W.QWEN3_OMNI, "fp8")
    assert dec8 == 544084992
