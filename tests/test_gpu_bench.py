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


def _check_roofline(rl, dtype):
    assert rl["bound"] in ("hbm", "mfma") and rl["unit"] in ("GB/s", "TFLOP/s")
    work = rl["algorithmic_bytes"] if rl["bound"] == "hbm" else rl["algorithmic_flops"]
    scale = 1e-3 if rl["bound"] == "hbm" else 1e-6
    assert rl["achieved"] == pytest.approx(work / rl["kernel_avg_us"] * scale, rel=1e-9)
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-12)


def test_default_line_times_every_config():
    """The default run times the largest workload (the 70B-shaped long suffix) and,
    in the same line, the other four configurations; the int8 one over its 32
    layers back to back, reported per layer."""
    say("bench.py (default workload and configs)")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--steps", "8",
                        "--warmup", "2", "--no-cpu-baseline"],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    assert KEYS <= set(d)
    assert d["config"]["workload"] == "70b-long-suffix-bf16"
    assert d["roofline"]["bound"] == "mfma" and d["roofline"]["kernel"] == "attn_paged"
    _check_roofline(d["roofline"], "bf16")
    cfgs = d["configs"]
    assert set(cfgs) == {"tiny-fp32", "llama3-8b-layer-bf16", "ragged-batch-bf16",
                         "int8-32layer"}
    for name, c in cfgs.items():
        assert c["config"]["workload"] == name and c["value"] > 0, name
        _check_roofline(c["roofline"], c["dtype"])
    c4 = cfgs["int8-32layer"]
    assert c4["config"]["layers"] == 32
    assert c4["ms_per_layer"] == pytest.approx(c4["ms_per_step"] / 32, rel=1e-12)
    assert c4["value"] == pytest.approx(8192 / (c4["ms_per_layer"] * 1e-3), rel=1e-9)
