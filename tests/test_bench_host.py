"""bench.py's host-side contract, on the CPU: one GPU only, and the
committed counter summaries it reads (traffic and vector issue per launch),
taken only when they match the kernel's sources, workload, batch and size."""
import glob
import json
import os
import re
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    msg = json.loads(p.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_summaries_are_read_only_for_their_sources(tmp_path):
    src = tmp_path / "kern.hip"
    src.write_text("// a kernel\n")
    h = bench.source_hash([str(src)])
    summary = tmp_path / "summary.md"
    summary.write_text(f"notes\n\ntraffic: {h} wl 1024 8 fetch_bytes=100 write_bytes=20\n"
                       f"issue: {h} wl 1024 8 valu_insts=4096 salu_insts=10 gui_active=8192\n")
    assert bench.measured_traffic("wl", 1024, 8, str(summary), [str(src)]) == 120
    iss = bench.measured_issue("wl", 1024, 8, str(summary), [str(src)])
    # 4096 instructions x 4 cycles over 1,024 SIMDs and 8192 / 8 cycles
    assert abs(iss["valu_busy"] - 4096 * 4 / (1024 * 1024)) < 1e-12
    assert bench.measured_traffic("wl", 2048, 8, str(summary), [str(src)]) is None
    assert bench.measured_traffic("wl", 1024, 16, str(summary), [str(src)]) is None
    src.write_text("// the kernel changed\n")
    assert bench.measured_traffic("wl", 1024, 8, str(summary), [str(src)]) is None
    assert bench.measured_issue("wl", 1024, 8, str(summary), [str(src)]) is None


def test_committed_summary_lines_parse():
    found = 0
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.md")):
        for line in open(path):
            if line.startswith("traffic:"):
                assert re.match(r"traffic: [0-9a-f]{16} \S+ \d+ \d+ fetch_bytes=\d+ write_bytes=\d+$",
                                line.strip()), (path, line)
                found += 1
            elif line.startswith("issue:"):
                assert re.match(r"issue: [0-9a-f]{16} \S+ \d+ \d+ valu_insts=\d+ salu_insts=\d+ "
                                r"gui_active=\d+$", line.strip()), (path, line)
                found += 1
    assert found >= 10


def test_cpu_baseline_legs_and_fields():
    """Both legs of the CPU baseline (all cores, one core) on consecutive
    candidates of a small batch, with the CPU model reported."""
    import workloads as W
    prob = W.make_problem(1)
    rows = W.generator_for(prob, 1).generate(0, 256)
    cpu = bench.cpu_oracle_baseline(prob, rows, 0.2)
    assert cpu["kind"] == "oracle" and cpu["unit"] == "candidates/s"
    assert cpu["cores"] >= 1 and cpu["value"] > 0 and cpu["one_core"]["value"] > 0
    assert cpu["ops_per_s"] == cpu["value"] * prob.n_total or abs(
        cpu["ops_per_s"] / (cpu["value"] * prob.n_total) - 1) < 1e-9
    assert isinstance(cpu["cpu_model"], str) and cpu["cpu_model"]


def test_oracle_timing_path():
    """--path oracle (no GPU work): one line with every workload's one-core
    and all-core oracle rates, the full sweep of the requested workloads, and
    the host description."""
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--path", "oracle",
                        "--n-cand", "32", "--oracle-full", "1"],
                       capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stderr[-2000:]
    rec = json.loads(p.stdout.strip().splitlines()[-1])
    assert rec["kind"] == "oracle" and rec["threads"] >= 1 and rec["cpu_model"]
    assert set(rec["workloads"]) == {"tiny", "vlm_s8", "vlm_interleaved_16x2", "diffusion_s32",
                                     "large_16x4"}
    for name, w in rec["workloads"].items():
        assert w["candidates"] == 32
        assert w["one_core"]["candidates_per_s"] > 0 and w["all_cores"]["candidates_per_s"] > 0
        assert ("full_sweep" in w) == (name == "tiny")
    assert rec["workloads"]["tiny"]["full_sweep"]["candidates"] == 1024
