"""Benchmark of the C2KV compose-and-attend hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 70b-long-suffix-bf16]

A step is one pass of the path over one layer of a synthetic workload:
c2kv_compose_attend (gather, decode, re-rotate, suffix RoPE, split-K attention
and merge) for the short-suffix workloads, c2kv_compose then c2kv_attend for
the long-suffix one.  The int8 workload's step is its 32 layers back to back,
each with its own independently seeded cache and suffix (one shared plan), and
reports per layer.  The plan (host layout, built once per batch of requests and
shared by all layers) is built and uploaded before the timed region.

The default workload is the largest single-GPU one (the 70B-shaped long
suffix); the same run also times the tiny fp32, Llama-3-8B layer, ragged batch
and 32-layer int8 workloads and reports them under "configs" in the same line
(--no-configs skips them).

Inputs live in HBM before timing starts.  Steps rotate over enough device
copies of the inputs that their footprint exceeds twice the 256 MB Infinity
Cache, so small workloads are timed against HBM rather than the cache.  The K
timed steps are replayed from a HIP graph (captured once over the copies);
an eager run with per-kernel HIP events gives the dominant kernel's average
duration for the roofline fraction.

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import synth  # noqa: E402  (seeded input generators; shapes of the workloads)

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "composed KV tokens attended/sec per layer + % HBM/MFMA roofline, 1 MI355X"
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E, GB/s
PEAK_BF16_TFLOPS = 2500.0       # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3        # fp32 (MFMA / packed vector)
MALL_BYTES = 256 << 20

WORKLOADS = {
    "tiny-fp32": 1,
    "llama3-8b-layer-bf16": 2,
    "ragged-batch-bf16": 3,
    "int8-32layer": 4,
    "70b-long-suffix-bf16": 5,
    "decode-32k-4x-bf16": 6,
    "decode-128k-4x-bf16": 7,
    "decode-128k-16x-bf16": 8,
    "decode-128k-1x-bf16": 9,
    "llama3-8b-layer-prerope-bf16": 10,
    "llama3-8b-layer-c2x4-bf16": 11,
    "llama3-8b-layer-host-zerocopy": 2,
    "llama3-8b-layer-host-load": 2,
    "int8-layer-host-zerocopy": 4,
    "int8-layer-host-load": 4,
    "sif-extract-llama3-8b-bf16": 0,
}
# decode steps over the rest of the context x compression grid (Section 4.3)
for _i, (_ctx, _r) in enumerate(synth.DECODE_GRID):
    WORKLOADS[f"decode-{_ctx}k-{_r}x-bf16"] = 12 + _i
# extraction-time attention with Structured Information Flow over document chunks
SIF = {"sif-extract-llama3-8b-bf16"}
DEFAULT_WORKLOAD = "70b-long-suffix-bf16"
# timed in the same run as the default workload, reported under "configs"
SECONDARY = ["tiny-fp32", "llama3-8b-layer-bf16", "ragged-batch-bf16", "int8-32layer"]
SECONDARY_STEPS, SECONDARY_WARMUP = 256, 16
LONG_SUFFIX = {"70b-long-suffix-bf16"}
# one generated token over a cache composed once beforehand: the step is c2kv_attend
DECODE = {name for name, idx in WORKLOADS.items() if 6 <= idx <= 9 or idx >= 12}
# the load step: chunks stored compressed in page-locked host memory, read in place by the
# fused kernel over the host link, or copied to the device first (c2kv_load)
HOST_ZEROCOPY = {"llama3-8b-layer-host-zerocopy", "int8-layer-host-zerocopy"}
HOST_LOAD = {"llama3-8b-layer-host-load", "int8-layer-host-load"}
PEAK_HOST_LINK_GBS = 64.0       # PCIe 5.0 x16, one direction


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_work(w, composed: np.ndarray):
    """Bytes and flops the method must move / compute for one layer (per launch
    of the attention kernel), excluding unread pool rows and masked pairs.

    bytes per composed token: K and V rows of one token (2 H_kv D b_kv), the
      int8 scales (2 H_kv 4) and the slot index (4);
    bytes per suffix token: q and out (2 H_q D b_act), suffix k and v
      (2 H_kv D b_act), lse (4 H_q);
    flops: 4 H_q D per visible (query, key) pair (Q K^T and P V)."""
    Hq, Hkv, D, S, B = w.n_q_heads, w.n_kv_heads, w.head_dim, w.suffix_len, w.batch
    b_kv = {"f32": 4, "bf16": 2, "i8": 1}[w.pool_dtype]
    b_act = {"f32": 4, "bf16": 2}[w.act_dtype]
    n_tok = int(composed.sum())
    per_tok = 2 * Hkv * D * b_kv + (8 * Hkv if w.pool_dtype == "i8" else 0) + 4
    per_q = 2 * Hq * D * b_act + 2 * Hkv * D * b_act + 4 * Hq
    byts = n_tok * per_tok + B * S * per_q
    pairs = n_tok * S + B * S * (S + 1) // 2
    flops = 4 * Hq * D * pairs
    return dict(bytes=int(byts), flops=int(flops), bytes_per_token=per_tok,
                bytes_per_query=per_q, pairs=int(pairs), tokens=n_tok)


def paged_attend_bytes(w, composed):
    """Attention over materialised pages reads act-dtype K/V rows."""
    b_act = {"f32": 4, "bf16": 2}[w.act_dtype]
    Hq, Hkv, D, S, B = w.n_q_heads, w.n_kv_heads, w.head_dim, w.suffix_len, w.batch
    n_tok = int(composed.sum())
    per_q = 2 * Hq * D * b_act + 2 * Hkv * D * b_act + 4 * Hq
    return n_tok * (2 * Hkv * D * b_act + 4) + B * S * per_q


def _code_only(text: str) -> str:
    """C++ source without comments and blank space: what the compiler sees."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_sha() -> str:
    """Hash of the code (comments and layout aside) of the kernels, the plan and the C ABI."""
    h = hashlib.sha256()
    for f in ("kernels.hip", "plan.cpp", "api.cpp"):
        with open(os.path.join(ROOT, "paper_2607_17715_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, kernel: str, n_launch_bytes: float):
    """HBM traffic per launch from the committed rocprofv3 counter summary, or
    None when there is none or the kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_sha") != kernel_source_sha():
        return None
    return t.get("hbm_bytes_per_launch")


def host_threads():
    """(cores this process may run on, the BLAS library's thread count)."""
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    return cores, blas


def cpu_baseline(w, idx: int):
    """The float64 oracle timed on this host on a bounded sample of the workload."""
    import oracle
    cores, blas = host_threads()
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx, w.seg_new_pos0)
    N = int(lay["composed_len"].sum())
    S = w.suffix_len
    if idx in (1, 2, 4) or idx >= 6:   # every workload but the two largest prefills
        # whole layer, repeated for about 10 s
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.compose_attend(w)
            reps += 1
            el = time.perf_counter() - t0
            if el > 10.0 or reps >= 5000:
                break
        per_layer = el / reps
        sample = f"whole layer x{reps} (compose of {N} slots + attention of all {S} suffix tokens)"
    else:
        # compose every kept token of the first request(s), attention of a few suffix rows,
        # repeated for about 10 s, scaled to the whole layer
        reqs = list(range(min(w.batch, 2)))
        rows = list(range(0, S, max(1, S // 8)))[:8]
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.compose_attend(w, rows=rows, requests=reqs)
            reps += 1
            el = time.perf_counter() - t0
            if el > 10.0 or reps >= 1000:
                break
        frac_req = float(lay["composed_len"][reqs].sum() + len(reqs)) / float(N + w.batch)
        per_layer = el / reps / frac_req * (S / len(rows))
        sample = (f"requests {reqs} ({int(lay['composed_len'][reqs].sum())} slots composed), "
                  f"{len(rows)} of {S} suffix rows, x{reps}; scaled by suffix rows and by slots")
    return {"value": N / per_layer, "unit": "tokens/s/layer", "cores": cores,
            "blas_threads": blas, "kind": "oracle", "sample": sample,
            "seconds_per_layer": per_layer}


def time_steps(step, copies, args, c2kv, torch, steps=None, warmup=None, launches_per_step=1):
    """Warm-up, an eager timing, the timed graph replays (K steps captured over the
    input copies), and a pass with per-kernel dispatch-stamped events.  Returns
    (ms per step, eager ms per step, per-kernel averages, whether graphs ran)."""
    K = args.steps if steps is None else steps
    for i in range(args.warmup if warmup is None else warmup):
        step(i)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ke = max(1, min(K, 256 // launches_per_step))
    torch.cuda.synchronize()
    start.record()
    for i in range(ke):
        step(i)
    end.record()
    torch.cuda.synchronize()
    eager_ms = start.elapsed_time(end) / ke
    graph_used = not args.no_graph
    if graph_used:
        n_full, rem = divmod(K, copies)
        g_full = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_full):
            for i in range(copies):
                step(i)
        g_rem = None
        if rem:
            g_rem = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_rem):
                for i in range(rem):
                    step(i)
        g_full.replay()
        torch.cuda.synchronize()
        start.record()
        for _ in range(n_full):
            g_full.replay()
        if g_rem is not None:
            g_rem.replay()
        end.record()
        torch.cuda.synchronize()
        total_ms = start.elapsed_time(end)
    else:
        torch.cuda.synchronize()
        start.record()
        for i in range(K):
            step(i)
        end.record()
        torch.cuda.synchronize()
        total_ms = start.elapsed_time(end)
    c2kv.timing_reset()
    c2kv.timing_enable(True)
    for i in range(ke):
        step(i)
    torch.cuda.synchronize()
    c2kv.timing_enable(False)
    kern = {}
    for name in ("compose", "attn_paged", "attn_pool", "merge"):
        ms, n = c2kv.timing_read(name)
        if n:
            kern[name] = {"avg_us": 1e3 * ms / n, "launches": n}
    c2kv.timing_reset()
    return total_ms / K, eager_ms, kern, graph_used


def run_sif(args, c2kv, synth, torch):
    """Extraction-time SIF attention: the value counts the tokens of the extraction
    sequences (originals and C^2 tokens) per second and layer."""
    import oracle
    w = synth.sif_config(args.workload)
    plan = c2kv.Plan.for_sif(w, kv_splits=args.kv_splits, rows_per_block=args.rows_per_block,
                             merge_mode=args.merge_mode).upload()
    B, L, Hq, Hkv, D = w.batch, w.seq_len, w.n_q_heads, w.n_kv_heads, w.head_dim
    b_act = 4 if w.act_dtype == "f32" else 2
    vis = oracle.sif_mask(w.n_tokens, w.block, w.sink)
    pairs = int(vis.sum()) * B
    byts = B * L * ((2 * Hq + 2 * Hkv) * D * b_act + 4 * Hq)     # q, k, v, out, lse
    flops = 4 * Hq * D * pairs
    base = dict(q=c2kv.to_device(w.q, w.act_dtype), k=c2kv.to_device(w.k, w.act_dtype),
                v=c2kv.to_device(w.v, w.act_dtype))
    footprint = sum(t.numel() * t.element_size() for t in base.values())
    copies = args.copies or int(min(64, max(2, math.ceil(2.2 * MALL_BYTES / footprint))))
    sets = [base] + [{k: t.clone() for k, t in base.items()} for _ in range(copies - 1)]
    for s in sets:
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty((B, Hq, L), dtype=torch.float32, device="cuda")

    def step(i):
        s = sets[i % copies]
        c2kv.c2kv_attend(plan, None, None, s["q"], s["k"], s["v"], s["out"], s["lse"])

    ms_per_step, eager_ms, kern, graph_used = time_steps(step, copies, args, c2kv, torch)
    assert torch.isfinite(sets[0]["out"]).all().item(), "non-finite output"
    dom_s = kern["attn_paged"]["avg_us"] * 1e-6
    t_hbm, t_mfma = byts / (PEAK_HBM_GBS * 1e9), flops / (PEAK_BF16_TFLOPS * 1e12)
    if t_hbm >= t_mfma:
        roof = {"bound": "hbm", "achieved": byts / dom_s / 1e9, "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": flops / dom_s / 1e12, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof.update(traffic=load_traffic(args.workload, "attn_paged", byts), kernel="attn_paged",
                kernel_avg_us=kern["attn_paged"]["avg_us"], algorithmic_bytes=byts,
                algorithmic_flops=flops)
    result = {
        "metric": METRIC, "value": B * L / (ms_per_step * 1e-3), "unit": "tokens/s/layer",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if w.act_dtype == "f32" else "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "n_q_heads": Hq, "n_kv_heads": Hkv,
                   "head_dim": D, "batch": B, "n_tokens": w.n_tokens, "block": w.block,
                   "sink": w.sink, "sequence_tokens": B * L,
                   "path": "SIF extraction attention (c2kv_attend with a SIF plan)",
                   "plan": {k: plan.info[k] for k in ("rows_per_block", "n_work_items",
                                                      "n_merge_groups", "max_splits")},
                   "input_copies": copies, "graph": graph_used},
        "roofline": roof, "kernels_us": kern, "eager_ms_per_step": eager_ms,
        "source_sha": kernel_source_sha(),
    }
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on the host (cpu_baseline)")
        t0 = time.perf_counter()
        reps = 0
        while True:
            q, k, v = (oracle.decode_storage(x[reps % B], w.act_dtype) for x in (w.q, w.k, w.v))
            oracle.sif_attend(q, k, v, w.n_tokens, w.block, w.sink, w.rope_base)
            reps += 1
            el = time.perf_counter() - t0
            if el > 10.0 or reps >= 4 * B:
                break
        cores, blas = host_threads()
        result["cpu_baseline"] = {"value": reps * L / el, "unit": "tokens/s/layer",
                                  "cores": cores, "blas_threads": blas, "kind": "oracle",
                                  "sample": f"{reps} whole sequences of {L} tokens"}
    print(json.dumps(result), flush=True)


def run_workload(name, args, c2kv, torch, steps, warmup, with_cpu):
    """Time one workload (not SIF); returns its result object (the JSON line's
    fields, without the headline-only keys)."""
    idx = WORKLOADS[name]
    log(f"workload {name}: generating inputs")
    sp = synth.spec(idx)
    w = synth.config(idx)
    layers = sp.layers if name == "int8-32layer" else 1
    host_mode = ("zerocopy" if name in HOST_ZEROCOPY else
                 "load" if name in HOST_LOAD else None)
    if host_mode:
        w = synth.compress_pool(w)
    plan = c2kv.Plan.for_workload(w, kv_splits=args.kv_splits,
                                  rows_per_block=args.rows_per_block,
                                  merge_mode=args.merge_mode).upload()
    composed, span_end = plan.requests()
    work = algorithmic_work(w, composed)
    long_suffix = name in LONG_SUFFIX
    decode = name in DECODE
    paged = long_suffix or decode
    act = torch.float32 if w.act_dtype == "f32" else torch.bfloat16

    def out_lse(s):
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty((w.batch, w.n_q_heads, w.suffix_len), dtype=torch.float32,
                               device="cuda")
        return s

    if layers > 1:
        # every layer its own seeded cache and suffix, drawn on the device; one plan
        sets = []
        for layer in range(layers):
            d = synth.int8_layer_device(sp, layer, synth.BASE_SEED + idx)
            d["ks"], d["vs"] = d.pop("k_scale"), d.pop("v_scale")
            d["pool"] = c2kv.pool_desc(d["k"], d["v"], d["ks"], d["vs"])
            sets.append(out_lse(d))
        torch.cuda.synchronize()
        copies = 1
        log(f"{layers} layers drawn on the device; the step runs them back to back")

        def step(i):
            for s in sets:
                c2kv.c2kv_compose_attend(plan, s["pool"], s["q"], s["k_suf"], s["v_suf"],
                                         s["out"], s["lse"])
    else:
        # ---- device inputs, replicated so the rotation spans > 2x the Infinity Cache
        base = dict(k=c2kv.to_device(w.pool_k, w.pool_dtype),
                    v=c2kv.to_device(w.pool_v, w.pool_dtype),
                    ks=None if w.pool_k_scale is None else c2kv.to_device(w.pool_k_scale, "f32"),
                    vs=None if w.pool_v_scale is None else c2kv.to_device(w.pool_v_scale, "f32"),
                    q=c2kv.to_device(w.q, w.act_dtype), k_suf=c2kv.to_device(w.k_suf, w.act_dtype),
                    v_suf=c2kv.to_device(w.v_suf, w.act_dtype))
        if paged:
            ksh, vsh = c2kv.page_shapes(plan)
        if decode:
            # the step reads the composed pages; each copy gets its own
            footprint = 2 * math.prod(ksh) * (4 if act == torch.float32 else 2)
        else:
            footprint = sum(t.numel() * t.element_size() for t in base.values() if t is not None)
        copies = args.copies or int(min(64, max(2, math.ceil(2.2 * MALL_BYTES / footprint))))
        log(f"footprint {footprint / 1e6:.1f} MB per copy, {copies} copies")
        if host_mode:
            # host memory is not cached on the device side: two copies, each with its
            # own device pool (the load destination)
            copies = args.copies or 2
            hosts = [c2kv.HostPool(w.pool_k, w.pool_v, w.pool_dtype, w.pool_k_scale,
                                   w.pool_v_scale) for _ in range(copies)]
            sets = [base] + [{k: (None if t is None else t.clone()) for k, t in base.items()}
                             for _ in range(copies - 1)]
            for s, h in zip(sets, hosts):
                s["host"] = h.desc
            log(f"host pools: {copies} x {hosts[0].nbytes / 1e6:.1f} MB page-locked")
        elif decode:
            sets = [dict(base) for _ in range(copies)]          # pool shared: composed once per copy
        else:
            sets = [base] + [{k: (None if t is None else t.clone()) for k, t in base.items()}
                             for _ in range(copies - 1)]
        for s in sets:
            s["pool"] = c2kv.pool_desc(s["k"], s["v"], s["ks"], s["vs"])
            out_lse(s)
        if long_suffix:
            kp = torch.empty(ksh, dtype=act, device="cuda")
            vp = torch.empty(vsh, dtype=act, device="cuda")
        if decode:
            for s in sets:
                s["kp"] = torch.empty(ksh, dtype=act, device="cuda")
                s["vp"] = torch.empty(vsh, dtype=act, device="cuda")
                c2kv.c2kv_compose(plan, s["pool"], s["kp"], s["vp"])
            torch.cuda.synchronize()
            log(f"composed {copies} page copies (untimed, as at prefill)")

        def step(i):
            s = sets[i % copies]
            if host_mode == "zerocopy":
                c2kv.c2kv_compose_attend(plan, s["host"], s["q"], s["k_suf"], s["v_suf"],
                                         s["out"], s["lse"])
            elif host_mode == "load":
                c2kv.c2kv_load(plan, s["host"], s["pool"])
                c2kv.c2kv_compose_attend(plan, s["pool"], s["q"], s["k_suf"], s["v_suf"],
                                         s["out"], s["lse"])
            elif decode:
                c2kv.c2kv_attend(plan, s["kp"], s["vp"], s["q"], s["k_suf"], s["v_suf"],
                                 s["out"], s["lse"])
            elif long_suffix:
                c2kv.c2kv_compose(plan, s["pool"], kp, vp)
                c2kv.c2kv_attend(plan, kp, vp, s["q"], s["k_suf"], s["v_suf"], s["out"],
                                 s["lse"])
            else:
                c2kv.c2kv_compose_attend(plan, s["pool"], s["q"], s["k_suf"], s["v_suf"],
                                         s["out"], s["lse"])

    ms_per_step, eager_ms, kern, graph_used = time_steps(step, copies, args, c2kv, torch,
                                                         steps=steps, warmup=warmup,
                                                         launches_per_step=layers)
    for s in sets:
        assert torch.isfinite(s["out"]).all().item(), "non-finite output"
    ms_per_layer = ms_per_step / layers
    value = work["tokens"] / (ms_per_layer * 1e-3)

    dom = "attn_paged" if paged else "attn_pool"
    dom_s = kern[dom]["avg_us"] * 1e-6
    mfma_bound = idx in (3, 5)
    if mfma_bound:
        peak = PEAK_FP32_TFLOPS if w.act_dtype == "f32" else PEAK_BF16_TFLOPS
        achieved = work["flops"] / dom_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak}
        dom_bytes = paged_attend_bytes(w, composed) if long_suffix else work["bytes"]
    else:
        dom_bytes = paged_attend_bytes(w, composed) if decode else work["bytes"]
        achieved = dom_bytes / dom_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
    roof["traffic"] = load_traffic(name, dom, dom_bytes)
    roof["kernel"] = dom
    roof["kernel_avg_us"] = kern[dom]["avg_us"]
    roof["algorithmic_bytes"] = dom_bytes
    roof["algorithmic_flops"] = work["flops"]
    compose_roof = None
    if "compose" in kern:
        # the gather / dequant / re-rotation / page write step on its own: kept rows read
        # in the storage dtype (and their scales), composed rows written in the
        # activation dtype
        b_pool = {"f32": 4, "bf16": 2, "i8": 1}[w.pool_dtype]
        b_act = {"f32": 4, "bf16": 2}[w.act_dtype]
        n_tok = int(composed.sum())
        c_bytes = n_tok * w.n_kv_heads * (2 * w.head_dim * (b_pool + b_act)
                                          + (8 if w.pool_dtype == "i8" else 0))
        c_s = kern["compose"]["avg_us"] * 1e-6
        compose_roof = {"bound": "hbm", "achieved": c_bytes / c_s / 1e9, "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": c_bytes / c_s / 1e9 / PEAK_HBM_GBS,
                        "traffic": load_traffic(name, "compose", c_bytes),
                        "kernel": "compose", "kernel_avg_us": kern["compose"]["avg_us"],
                        "algorithmic_bytes": c_bytes}

    result = {
        "value": value,
        "unit": "tokens/s/layer",
        "ms_per_step": ms_per_step,
        "dtype": "f32" if w.act_dtype == "f32" else "bf16",
        "config": {"workload": name, "n_q_heads": w.n_q_heads,
                   "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "pool_dtype": w.pool_dtype, "batch": w.batch, "suffix_len": w.suffix_len,
                   "composed_tokens": work["tokens"], "layers": layers,
                   "path": ("attend over composed pages" if decode else
                            "compose+attend" if long_suffix else "compose_attend"),
                   "plan": {**{k: plan.info[k] for k in ("rows_per_block", "n_work_items",
                                                         "n_merge_groups", "max_splits")},
                            "merge_mode": args.merge_mode},
                   "input_copies": copies, "graph": graph_used},
        "roofline": roof,
        **({"compose_roofline": compose_roof} if compose_roof else {}),
        "kernels_us": kern,
        "eager_ms_per_step": eager_ms,
    }
    if layers > 1:
        result["ms_per_layer"] = ms_per_layer
    if host_mode:
        link = hosts[0].nbytes                  # every stored row of the compressed chunks
        result["host_link"] = {"bytes": link, "achieved": link / (ms_per_step * 1e-3) / 1e9,
                               "peak": PEAK_HOST_LINK_GBS, "unit": "GB/s",
                               "frac": link / (ms_per_step * 1e-3) / 1e9 / PEAK_HOST_LINK_GBS,
                               "path": ("kernel reads over the host link" if host_mode == "zerocopy"
                                        else "copy engines, then the fused kernel")}
        result["config"]["path"] = result["config"]["path"] + f" (pool in host memory, {host_mode})"
    if with_cpu:
        log("timing the float64 oracle on the host (cpu_baseline)")
        result["cpu_baseline"] = cpu_baseline(w, idx)
    return result


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1024)
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--copies", type=int, default=0, help="input copies to rotate over (0: auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="time only --workload (by default the default workload's run also "
                         "times the other configurations)")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--kv-splits", type=int, default=0)
    ap.add_argument("--rows-per-block", type=int, default=0)
    ap.add_argument("--merge-mode", type=int, default=0)
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one device copy of this many MiB first (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the compose-and-attend path here runs on a single "
              "MI355X (--gpus 1); sharding over several GPUs is not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_17715_amd as c2kv

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {n} bytes done")
        del src, dst

    if args.workload in SIF:
        return run_sif(args, c2kv, synth, torch)
    r = run_workload(args.workload, args, c2kv, torch, args.steps, args.warmup,
                     with_cpu=not args.no_cpu_baseline)
    result = {
        "metric": METRIC,
        "value": r.pop("value"),
        "unit": r.pop("unit"),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": r.pop("dtype"),
        "data": "synthetic",
        **r,
        "source_sha": kernel_source_sha(),
    }
    if args.workload == DEFAULT_WORKLOAD and not args.no_configs:
        # the other configurations, in the same run: their per-layer figures and the
        # dominant kernel's roofline (inputs freed between them)
        cfgs = {}
        for name in SECONDARY:
            torch.cuda.empty_cache()
            cfgs[name] = run_workload(name, args, c2kv, torch, SECONDARY_STEPS,
                                      SECONDARY_WARMUP, with_cpu=False)
            cfgs[name]["steps"], cfgs[name]["warmup"] = SECONDARY_STEPS, SECONDARY_WARMUP
        result["configs"] = cfgs
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
