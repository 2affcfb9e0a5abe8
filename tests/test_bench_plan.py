"""Host-side checks of bench.py's timing arithmetic (no GPU): every timed
launch is part of a whole graph replay, exactly K launches per window, the
rotating operand pairs, and the trace summary's choice of timed dispatches."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("steps", [1, 2, 5, 20, 22, 64, 511, 512, 513, 1024, 1500, 20000])
def test_graph_plan_covers_exactly_the_steps(steps):
    ga, reps, rem = bench.graph_plan(steps)
    assert 1 <= ga <= bench.GRAPH_MAX and reps >= 1 and 0 <= rem < ga
    assert ga * reps + rem == steps
    if steps <= bench.GRAPH_MAX:
        assert (ga, reps, rem) == (steps, 1, 0)     # one replay of one graph, no eager launch


class _W:
    def __init__(self, algo):
        self.algo_bytes = algo


def test_operand_pairs():
    # >= 1 GiB of traffic where the window has enough launches, at most 64 pairs
    assert bench.operand_pairs(_W(50331648)) == 22                 # GELU 4096 x 3072 bf16
    assert bench.operand_pairs(_W(50331648), 20) == 20             # a 20-launch window uses 20
    assert bench.operand_pairs(_W(65536)) == 64
    assert bench.operand_pairs(_W(1 << 31)) == 2
    assert bench.operand_pairs(_W(50331648), 1) == 1


def test_trace_summary_takes_the_timed_half(tmp_path):
    # two windows; in each, 3 untimed dispatches of 100 ns then 3 + 6 timed of
    # 40 ns (and one dispatch outside every window that must be ignored)
    rows, wins, t = [], [], 1_000_000
    rows.append(("k", t - 500_000, t - 499_000))
    for _ in range(2):
        w0 = t
        for d in (100, 100, 100) + (40,) * 9:
            rows.append(("k", t, t + d))
            t += 1000
        wins.append([w0 - 10, 0, t + 10, 0])   # [boot start, mono start, boot end, mono end]
        t += 100_000
    csvp = tmp_path / "kernel_trace.csv"
    with open(csvp, "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        for n, a, b in rows:
            f.write("%s,%d,%d\n" % (n, a, b))
    winp = tmp_path / "w.json"
    winp.write_text(json.dumps({"lab:quake2": {"steps": 3, "algo_bytes": 400, "windows": wins}}))
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--summarize-trace",
                          str(csvp), "--trace-windows", str(winp)], capture_output=True, text=True,
                         check=True).stdout
    line = [ln for ln in out.splitlines() if ln.startswith("| lab:quake2")][0]
    cells = [c.strip() for c in line.strip("|").split("|")]
    assert cells[2] == "18" and float(cells[3]) == 40.0 and cells[5] == "40" and cells[6] == "40"
    assert float(cells[7]) == 10.0                       # 400 bytes / 40 ns
    assert float(cells[9]) == 1000.0                     # starts 1000 ns apart


def test_attention_config_filter_parses(monkeypatch):
    """--attn-config selects one heads x seq shape and optionally one mask of
    the attention section (used for counter passes)."""
    monkeypatch.setattr(sys, "argv", ["bench.py", "--section", "attention",
                                      "--attn-config", "32x2048:noncausal"])
    a = bench.parse()
    assert a.section == "attention" and a.attn_config == "32x2048:noncausal"
    shape, _, mask = a.attn_config.partition(":")
    assert tuple(int(v) for v in shape.split("x")) == (32, 2048) and mask == "noncausal"
