"""Per-kernel timing through the C ABI: with timing on, each launch of each
kernel is counted under its name with a positive duration; reset clears the
counts; with timing off nothing is recorded; results are unchanged by it."""
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, say

pytestmark = pytest.mark.gpu


def test_timing_counts_every_launch():
    say("kernel timing")
    w = synth.small(batch=2, n_q_heads=16, n_kv_heads=4, suffix_len=40)
    dev = Dev(w)
    plan = c2kv.Plan.for_workload(w, kv_splits=3).upload()
    assert plan.info["n_merge_groups"] > 0
    ksh, vsh = c2kv.page_shapes(plan)
    kp = torch.empty(ksh, dtype=torch.bfloat16, device="cuda")
    vp = torch.empty(vsh, dtype=torch.bfloat16, device="cuda")

    def run(out):
        c2kv.c2kv_compose_attend(plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out, None)
        c2kv.c2kv_compose(plan, dev.pool, kp, vp)
        c2kv.c2kv_attend(plan, kp, vp, dev.q, dev.k_suf, dev.v_suf, out, None)

    ref = dev.out_like()
    run(ref)
    torch.cuda.synchronize()
    try:
        c2kv.timing_reset()
        c2kv.timing_enable(True)
        out = dev.out_like()
        for _ in range(3):
            run(out)
        torch.cuda.synchronize()
        want = {"attn_pool": 3, "compose": 3, "attn_paged": 3, "merge": 6}
        for name, n in want.items():
            ms, launches = c2kv.timing_read(name)
            say(f"{name}: {launches} launches, {ms:.4f} ms")
            assert launches == n and ms > 0.0, (name, launches, ms)
        assert torch.equal(out, ref)
        c2kv.timing_reset()
        assert c2kv.timing_read("attn_pool") == (0.0, 0)
        c2kv.timing_enable(False)
        run(out)
        torch.cuda.synchronize()
        assert c2kv.timing_read("attn_pool") == (0.0, 0)
        assert c2kv.timing_read("no such kernel") == (0.0, 0)
    finally:
        c2kv.timing_enable(False)
        c2kv.timing_reset()
