"""Host logic of bench.py, on the CPU: the one-GPU guard, the algorithmic byte
and flop counts behind the roofline, the code hash that ties counter summaries
to the kernels, and the workload names against their recipes."""
import os
import subprocess
import sys

import numpy as np

import bench
import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_work_counts_pairs_and_bytes():
    """Per request: every suffix token t sees the N_b composed slots and suffix
    tokens 0..t; each composed token moves its K and V rows (and int8 scales)
    and a slot index, each suffix token its q, out, k, v rows and lse."""
    for pool_dtype in ("bf16", "i8", "f32"):
        w = synth.small(pool_dtype=pool_dtype, batch=3, keep=("ratio", 0.1, 0.7))
        lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                    w.seg_kept_off, w.kept_idx, w.seg_new_pos0)
        composed = np.asarray(lay["composed_len"], np.int64)
        got = bench.algorithmic_work(w, composed)
        S, Hq, Hkv, D = w.suffix_len, w.n_q_heads, w.n_kv_heads, w.head_dim
        pairs = 0
        for n_b in composed:
            for t in range(S):
                pairs += int(n_b) + t + 1
        assert got["pairs"] == pairs
        assert got["flops"] == 4 * Hq * D * pairs
        b_kv = {"f32": 4, "bf16": 2, "i8": 1}[pool_dtype]
        b_act = 4 if pool_dtype == "f32" else 2
        byts = 0
        for n_b in composed:
            for _ in range(int(n_b)):
                byts += 2 * Hkv * D * b_kv + 4 + (2 * Hkv * 4 if pool_dtype == "i8" else 0)
            for _ in range(S):
                byts += 2 * Hq * D * b_act + 2 * Hkv * D * b_act + Hq * 4
        assert got["bytes"] == byts, pool_dtype


def test_code_hash_ignores_comments_and_layout():
    a = "int f(int x) {\n  return x + 1;  // one more\n}\n/* block\n comment */"
    b = "int f(int x) { return x + 1; }"
    c = "int f(int x) { return x + 2; }"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(b) != bench._code_only(c)
    assert len(bench.kernel_source_sha()) == 16


def test_workload_names_match_their_recipes():
    for name, idx in bench.WORKLOADS.items():
        if name in bench.SIF:
            continue
        sp = synth.spec(idx)
        if name in bench.HOST_ZEROCOPY | bench.HOST_LOAD:
            assert sp.name.split("-")[0] == name.split("-")[0]
            continue
        assert sp.name == name
        if name in bench.DECODE:
            ctx, r = name.split("-")[1:3]
            ctx, r = int(ctx[:-1]) * 1024, int(r[:-1])
            assert sp.suffix_len == 1 and sp.batch == 1
            assert sp.chunks_per_req * sp.chunk_len == ctx, name
            kept = sp.chunk_len if sp.keep == ("all",) else sp.keep[1]
            assert sp.keep[0] in ("all", "count") and kept * r == sp.chunk_len, name
    assert bench.DEFAULT_WORKLOAD in bench.WORKLOADS


def test_default_is_the_largest_config_and_the_rest_ride_along():
    """The headline is the largest single-GPU workload (most flops per layer); the
    other four configurations are timed in the same run."""
    flops = {}
    for name in [bench.DEFAULT_WORKLOAD] + bench.SECONDARY:
        sp = synth.spec(bench.WORKLOADS[name])
        kept = sp.keep[1] if sp.keep[0] == "count" else sp.chunk_len * sp.keep[2]
        n_tok = sp.batch * (sp.prefix_len + sp.chunks_per_req * kept)
        flops[name] = 4 * sp.n_q_heads * sp.head_dim * n_tok * sp.suffix_len
    assert max(flops, key=flops.get) == bench.DEFAULT_WORKLOAD == "70b-long-suffix-bf16"
    assert sorted(bench.WORKLOADS[n] for n in bench.SECONDARY) == [1, 2, 3, 4]
    assert synth.spec(bench.WORKLOADS["int8-32layer"]).layers == 32


def test_cpu_baseline_reports_host_cores():
    cores, blas = bench.host_threads()
    assert cores == len(os.sched_getaffinity(0)) and cores >= 1
    assert blas is None or blas >= 1
