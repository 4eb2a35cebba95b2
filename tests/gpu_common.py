"""Shared helpers of the GPU parity tests: move a synthetic workload to the
device, run the HIP path through the C ABI, and compare with the oracle.

Tolerances (the bar of the parity tests):
  * indices, layout, page placement: bit-exact;
  * fp32 workloads: max |gpu - oracle| <= 1e-5 on outputs;
  * bf16 / int8 workloads (unit-variance inputs): max <= 2e-2, mean <= 1e-2.
  * lse: fp32 1e-5; bf16 / int8 max <= 5e-2, mean <= 1e-2.  A score's error is
    dominated by the bf16 rounding of the scaled query and of the turned key
    (2^-9 relative each): |ds| <= |q||k| scale 2^-8, about 0.04 for the largest
    |q||k|/sqrt(128) ~ 11 of these inputs, and lse moves by at most max |ds|.
"""
import sys

import numpy as np
import torch

import oracle
import paper_2607_17715_amd as c2kv

TOL = {
    "f32": dict(max=1e-5, mean=1e-5, lse_max=1e-5, lse_mean=1e-5),
    "bf16": dict(max=2e-2, mean=1e-2, lse_max=5e-2, lse_mean=1e-2),
}


def say(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


class Dev:
    """Device copies of one workload layer."""

    def __init__(self, w):
        self.w = w
        self.k = c2kv.to_device(w.pool_k, w.pool_dtype)
        self.v = c2kv.to_device(w.pool_v, w.pool_dtype)
        self.ks = None if w.pool_k_scale is None else c2kv.to_device(w.pool_k_scale, "f32")
        self.vs = None if w.pool_v_scale is None else c2kv.to_device(w.pool_v_scale, "f32")
        self.q = c2kv.to_device(w.q, w.act_dtype)
        self.k_suf = c2kv.to_device(w.k_suf, w.act_dtype)
        self.v_suf = c2kv.to_device(w.v_suf, w.act_dtype)
        self.pool = c2kv.pool_desc(self.k, self.v, self.ks, self.vs)

    def out_like(self):
        return torch.empty_like(self.q)

    def lse_like(self):
        B, S, Hq, _ = self.q.shape
        return torch.empty((B, Hq, S), dtype=torch.float32, device="cuda")


def run_fused(w, dev=None, plan=None, **opts):
    dev = dev or Dev(w)
    plan = plan or c2kv.Plan.for_workload(w, **opts).upload()
    out, lse = dev.out_like(), dev.lse_like()
    c2kv.c2kv_compose_attend(plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out, lse)
    torch.cuda.synchronize()
    return out, lse, plan, dev


def run_paged(w, dev=None, plan=None, **opts):
    dev = dev or Dev(w)
    plan = plan or c2kv.Plan.for_workload(w, **opts).upload()
    ks, vs = c2kv.page_shapes(plan)
    act = torch.float32 if w.act_dtype == "f32" else torch.bfloat16
    kp = torch.full(ks, float("nan"), dtype=act, device="cuda")
    vp = torch.full(vs, float("nan"), dtype=act, device="cuda")
    T = plan.info["total_slots"]
    src = torch.full((max(T, 1),), -7, dtype=torch.int64, device="cuda")
    pos = torch.full((max(T, 1),), -7, dtype=torch.int32, device="cuda")
    bt = torch.full((plan.info["batch"], plan.info["max_pages"]), -7, dtype=torch.int32,
                    device="cuda")
    c2kv.c2kv_compose(plan, dev.pool, kp, vp, src, pos, bt)
    out, lse = dev.out_like(), dev.lse_like()
    c2kv.c2kv_attend(plan, kp, vp, dev.q, dev.k_suf, dev.v_suf, out, lse)
    torch.cuda.synchronize()
    return out, lse, plan, dev, dict(k_pages=kp, v_pages=vp, src=src[:T], pos=pos[:T], bt=bt)


def compare(w, out, lse, ref_out, ref_lse, rows=None, what=""):
    """Element-wise comparison against the oracle (rows: suffix positions the
    oracle computed; default all)."""
    tol = TOL["f32" if w.act_dtype == "f32" else "bf16"]
    o = c2kv.to_numpy_f64(out)
    l = lse.detach().cpu().numpy().astype(np.float64)
    if rows is not None:
        o = o[:, rows]
        l = l[:, :, rows]
    assert np.isfinite(o).all(), f"{what}: non-finite output"
    err = np.abs(o - ref_out)
    lerr = np.abs(l - ref_lse)
    stats = dict(max=float(err.max()), mean=float(err.mean()), lse_max=float(lerr.max()),
                 lse_mean=float(lerr.mean()))
    say(f"{what} errors {stats}")
    assert stats["max"] <= tol["max"], (what, stats)
    assert stats["mean"] <= tol["mean"], (what, stats)
    assert stats["lse_max"] <= tol["lse_max"], (what, stats)
    assert stats["lse_mean"] <= tol["lse_mean"], (what, stats)
    return stats


def oracle_ref(w, rows=None, requests=None):
    out, lse, lay = oracle.compose_attend(w, rows=rows, requests=requests)
    return out, lse, lay
