"""bench.py's output line on the GPU: every field of the JSON contract, with the
roofline figures consistent among themselves (achieved = algorithmic work per
launch over the kernel's average duration; frac = achieved / peak)."""
import json
import os
import subprocess
import sys

import pytest

from gpu_common import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KEYS = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
        "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline"}


@pytest.mark.parametrize("workload,dtype", [("llama3-8b-layer-bf16", "bf16"),
                                            ("tiny-fp32", "f32")])
def test_bench_line_keeps_the_contract(workload, dtype):
    say(f"bench.py --workload {workload}")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload",
                        workload, "--steps", "16", "--warmup", "2", "--no-cpu-baseline"],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    assert KEYS <= set(d), KEYS - set(d)
    assert d["n_gpus"] == 1 and d["steps"] == 16 and d["warmup"] == 2
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["dtype"] == dtype and d["data"] == "synthetic" and d["vs_baseline"] is None
    assert d["config"]["workload"] == workload
    rl = d["roofline"]
    assert rl["bound"] in ("hbm", "mfma") and rl["unit"] in ("GB/s", "TFLOP/s")
    work = rl["algorithmic_bytes"] if rl["bound"] == "hbm" else rl["algorithmic_flops"]
    scale = 1e-3 if rl["bound"] == "hbm" else 1e-6      # per µs -> GB/s or TFLOP/s
    assert rl["achieved"] == pytest.approx(work / rl["kernel_avg_us"] * scale, rel=1e-9)
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-12)
    assert rl["peak"] == (8000.0 if rl["bound"] == "hbm" else
                          (2500.0 if dtype == "bf16" else 157.3))
