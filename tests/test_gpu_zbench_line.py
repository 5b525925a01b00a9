"""bench.py's output line on a real GPU: every field of the contract, on the
small workload (1 layer of 4 query heads over 1024 tokens) so that it runs in
seconds.  The committed counter summaries belong to the 128k workload, so
this line must carry no traffic figure."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_contract():
    print("[bench contract] workload c1", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "c1",
                        "--steps", "3", "--warmup", "1", "--dense-reps", "1",
                        "--cpu-budget-s", "1"],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [x for x in r.stdout.splitlines() if x.strip()]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "ms/layer" and d["higher_is_better"] is False
    assert d["value"] > 0 and d["value"] == d["ms_per_step"]
    assert d["scaling"] == "weak" and d["vs_baseline"] is None
    assert d["dtype"] == "bf16" and d["data"] == "synthetic"
    c = d["config"]
    assert "workload" in c and c["seq_len"] == 1024 and c["n_q_heads"] == 4
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2500.0
    assert 0 < rf["achieved"] and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert rf["traffic"] is None and d["mfma_busy_counter"] is None
    pf = d["probe_select_fused"]
    assert pf["bitwise_equal_to_separate"] is True and pf["ms"] > 0
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1
    assert cb["unit"] == "ms/layer" and cb["sample"]
