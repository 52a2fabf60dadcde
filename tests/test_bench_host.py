"""Host-side logic of bench.py: the kernel-source hash that ties a committed
HBM-traffic summary to the code it was measured on (no GPU needed)."""
import os
import shutil

import numpy as np

import bench

SRC = os.path.join(os.path.dirname(bench.__file__), "paper_2609_09721_amd", "csrc", "efq_attn.hip")


def _copy(tmp_path, edit=None):
    text = open(SRC).read()
    if edit:
        text = edit(text)
    p = tmp_path / "k.hip"
    p.write_text(text)
    return str(p)


def test_hash_ignores_comments_and_blank_lines(tmp_path):
    h = bench.kernel_hash(_copy(tmp_path))
    assert h == bench.kernel_hash()
    assert bench.kernel_hash(_copy(tmp_path, lambda t: "// a new note\n\n" + t)) == h
    def block(t):
        assert "constexpr int kBarPhases = 4;" in t
        return t.replace("constexpr int kBarPhases = 4;",
                         "/* a block\n   comment */ constexpr int kBarPhases = 4;  // note", 1)
    assert bench.kernel_hash(_copy(tmp_path, block)) == h


def test_hash_changes_with_code(tmp_path):
    h = bench.kernel_hash()
    edited = _copy(tmp_path, lambda t: t.replace("constexpr int kBarPhases = 4;",
                                                 "constexpr int kBarPhases = 2;", 1))
    assert bench.kernel_hash(edited) != h


def test_traffic_only_for_matching_source(tmp_path):
    d = tmp_path / "profiles"
    d.mkdir()
    f = d / "attn_fwd_w_traffic.txt"
    f.write_text(f"# summary\ntraffic_bytes_per_launch = 123456\nkernel_hash = {bench.kernel_hash()}\n")
    assert bench.read_traffic("w", str(d)) == 123456.0
    f.write_text("traffic_bytes_per_launch = 123456\nkernel_hash = 0000000000000000\n")
    assert bench.read_traffic("w", str(d)) is None
    assert bench.read_traffic("missing", str(d)) is None


def test_trace_and_counter_views_only_for_matching_source(tmp_path):
    d = tmp_path / "profiles"
    d.mkdir()
    h = bench.kernel_hash()
    (d / "attn_pp_kernel_w_stats.txt").write_text(
        f"# trace\nefq_calls = 3\nefq_avg_us = 5400.0\nefq_median_us = 5350.0\nkernel_hash = {h}\n")
    assert bench.read_trace_avg_ms("w", str(d)) == (5.4, 5.35)
    (d / "attn_pp_kernel_w_counters.txt").write_text(
        "valu_active_cycles_efq = 600\nvalu_active_cycles_expq = 900\n"
        f"valu_active_cycles_noop = 100\nkernel_hash = {h}\n")
    c = bench.read_stage_counters("w", str(d))
    assert (c["efq"], c["expq"]) == (500, 800) and c["speedup"] == round(1 - 500 / 800, 4)
    for f in d.iterdir():
        f.write_text(f.read_text().replace(h, "0000000000000000"))
    assert bench.read_trace_avg_ms("w", str(d)) is None
    assert bench.read_stage_counters("w", str(d)) is None


def test_committed_summaries_describe_the_committed_kernel():
    # the trace, counter, traffic and phase-stamp summaries under profiles/ were measured
    # on the kernel source as committed: bench.py reports their figures only
    # while the hash matches, so a kernel change without new summaries would
    # silently drop them from the measurement line
    d = os.path.join(os.path.dirname(bench.__file__), "profiles")
    h = bench.kernel_hash()
    for name in ("attn_pp_kernel_qwen3_8b_32k_stats.txt", "attn_pp_kernel_qwen3_8b_32k_counters.txt",
                 "attn_fwd_qwen3_8b_32k_traffic.txt", "attn_pp_kernel_qwen3_8b_32k_phases.txt"):
        lines = open(os.path.join(d, name)).read().splitlines()
        assert f"kernel_hash = {h}" in lines, name
    assert bench.read_trace_avg_ms("qwen3_8b_32k", d) is not None
    assert bench.read_stage_counters("qwen3_8b_32k", d) is not None
    assert bench.read_traffic("qwen3_8b_32k", d) is not None
    assert bench.read_stage_stamps("qwen3_8b_32k", d) is not None


def test_stamp_summary_round_trip(tmp_path):
    # the phase-stamp summary that paper_2609_09721_amd.phases writes is read
    # back by bench.py only while it carries the current kernel hash
    from paper_2609_09721_amd import phases
    res = {k: {"ms": 1.0, "M": {"median": m, "mean": m, "p90": m, "wait_median": 10.0,
                                "wait_mean": 10.0, "n": 1},
               "V": {"median": v, "mean": v, "p90": v, "wait_median": 20.0, "wait_mean": 20.0,
                     "n": 1}}
           for k, m, v in (("efq", 1200.0, 600.0), ("expq", 1400.0, 900.0),
                           ("lut", 1300.0, 650.0), ("noop", 700.0, 200.0))}
    d = tmp_path / "profiles"
    d.mkdir()
    text = phases.summarize(res, "w", "cmd", bench.kernel_hash())
    (d / "attn_pp_kernel_w_phases.txt").write_text(text)
    got = bench.read_stage_stamps("w", str(d))
    assert got["efq"] == 900 and got["expq"] == 1400
    assert got["speedup"] == round(1 - 900 / 1400, 4)
    assert "sclk_ghz" not in got                      # no clock pairs in res
    res["efq"]["sclk"] = 2.0834
    (d / "attn_pp_kernel_w_phases.txt").write_text(phases.summarize(res, "w", "cmd",
                                                                    bench.kernel_hash()))
    assert bench.read_stage_stamps("w", str(d))["sclk_ghz"] == 2.083
    (d / "attn_pp_kernel_w_phases.txt").write_text(text.replace(bench.kernel_hash(), "0" * 16))
    assert bench.read_stage_stamps("w", str(d)) is None


def test_stamp_clock_pairs():
    # (s_memtime, s_memrealtime) at a wave's first and last stamped phase end:
    # 2.1e6 shader ticks over 1e5 ticks of the 100 MHz counter is 2.1 GHz;
    # waves with no clock pair (zeros) are left out of the median
    from paper_2609_09721_amd import phases
    clk = np.zeros((4, 2, 4), dtype=np.int64)
    clk[:3, :, 0], clk[:3, :, 1] = 1000, 500
    clk[:3, :, 2], clk[:3, :, 3] = 1000 + 2_100_000, 500 + 100_000
    clk[0, 0, 2] = 1000 + 1_900_000
    assert abs(phases.sclk_ghz(clk) - 2.1) < 1e-12
