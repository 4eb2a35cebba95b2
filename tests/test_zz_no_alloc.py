"""The allocation-free entry point (c2kv_compose_attend_static) against
c2kv_compose_attend, through the C ABI.

Both run the same kernels; the static one takes its tables and split partials
from the library's static device array instead of a caller workspace.  Two
calls in a row share that array, the second with a smaller input, so the second
must not depend on what the first left there.  Results must be identical bit for
bit (outputs and LSE), and match the oracle to the parity bar.
"""
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, compare, oracle_ref, say

pytestmark = pytest.mark.gpu


def _static_vs_workspace(w, what, **opts):
    dev = Dev(w)
    ref_plan = c2kv.Plan.for_workload(w, **opts).upload()
    plan = c2kv.Plan.for_workload(w, **opts)            # never uploaded
    assert plan.info["workspace_bytes"] <= c2kv.STATIC_SCRATCH_BYTES
    out_ref, lse_ref = dev.out_like(), dev.lse_like()
    say(f"{what}: compose_attend with a workspace {opts}")
    c2kv.c2kv_compose_attend(ref_plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out_ref, lse_ref)
    out, lse = dev.out_like(), dev.lse_like()
    out.fill_(float("nan"))
    lse.fill_(float("nan"))
    say(f"{what}: compose_attend_static {opts} "
        f"(workspace {plan.info['workspace_bytes']} B, merges {plan.info['n_merge_groups']})")
    c2kv.c2kv_compose_attend_static(plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out, lse)
    torch.cuda.synchronize()
    assert torch.equal(out, out_ref), what
    assert torch.equal(lse, lse_ref), what
    return out, lse, plan


def test_static_scratch_two_calls_second_smaller():
    big = synth.config(2)                                   # Llama-3-8B layer: 144 split partials
    small = synth.small(pool_dtype="i8", batch=2, suffix_len=23)
    p_big = _static_vs_workspace(big, "llama3-8b-layer")[2]
    out, lse, p_small = _static_vs_workspace(small, "small int8")
    assert p_small.info["workspace_bytes"] < p_big.info["workspace_bytes"]
    assert p_big.info["n_merge_groups"] > 0 and p_small.info["n_merge_groups"] > 0
    ref_out, ref_lse, _ = oracle_ref(small)
    compare(small, out, lse, ref_out, ref_lse, what="small int8/static")


def test_static_scratch_in_kernel_merge_counters_restart():
    """With the in-kernel merge the array holds the splits' arrival counters;
    each call starts them from zero, so back-to-back calls agree."""
    w = synth.small(batch=2, suffix_len=40)
    for i in range(2):
        _static_vs_workspace(w, f"in-kernel merge, call {i}", merge_mode=1, kv_splits=3)
