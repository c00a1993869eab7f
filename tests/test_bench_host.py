"""CPU tests of bench.py's host logic around the committed counter figures: the scan's
HBM traffic is reported only while the kernel's code is the one the counters were
taken on, and only for the workload they were taken on; the score-only ablation's
dispatches are told apart from the scan's by their template arguments."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

SOURCE = os.path.join(bench.CSRC, "topk_kernels.hip")


def _scan_section_copy(tmp_path, name, edit):
    text = open(SOURCE).read()
    a = text.index(bench.SCAN_BEGIN)
    b = text.index(bench.SCAN_END)
    d = tmp_path / name
    d.mkdir()
    (d / "topk_kernels.hip").write_text(text[:a] + edit(text[a:b]) + text[b:])
    return str(d)


def test_digest_ignores_comments_and_blank_lines_not_code(tmp_path, monkeypatch):
    base = bench.scan_source_digest()
    first_nl = lambda s: s.index("\n") + 1  # noqa: E731
    commented = _scan_section_copy(tmp_path, "commented", lambda s: s[:first_nl(s)] + "// a note\n\n   // another\n" +
                                   s[first_nl(s):])
    monkeypatch.setattr(bench, "CSRC", commented)
    assert bench.scan_source_digest() == base
    changed = _scan_section_copy(tmp_path, "changed", lambda s: s.replace("constexpr int SCAN_KT = 64;",
                                                                          "constexpr int SCAN_KT = 64;  \nint unused_x;", 1))
    monkeypatch.setattr(bench, "CSRC", changed)
    assert bench.scan_source_digest() != base


def test_traffic_is_reported_only_for_its_kernel_and_workload(tmp_path, monkeypatch):
    got = bench.traffic_for_current_kernel("c3", 1)
    assert got is not None and got > 1.34e8  # at least the compulsory Q + K reads of one launch
    assert bench.traffic_for_current_kernel("c4", 1) is None  # another workload
    assert bench.traffic_for_current_kernel("c3", 4) is None  # not the fused scan
    changed = _scan_section_copy(tmp_path, "changed", lambda s: s.replace("constexpr int SCAN_KT = 64;",
                                                                          "constexpr int SCAN_KT = 64;\nint unused_x;", 1))
    monkeypatch.setattr(bench, "CSRC", changed)
    assert bench.traffic_for_current_kernel("c3", 1) is None  # the kernel's code changed


def test_score_only_ablation_is_told_apart():
    name = "void topk::k_fused_scan<%s>(topk::ScanArgs)"
    assert bench._is_scan_ablation(name % "64, 11, 2, false, true, 20, false")
    assert not bench._is_scan_ablation(name % "64, 11, 2, false, false, 20, false")
    assert not bench._is_scan_ablation(name % "128, 3, 2, true, false, 0, true")  # direct mode
    assert not bench._is_scan_ablation("void topk::k_cand_select<false>(topk::Problem)")
