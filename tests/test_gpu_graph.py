"""The C ABI's launches inside a captured HIP graph: every replay, with eager
work of the same plan interleaved, reproduces the eager result bit for bit."""
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("opts", [dict(), dict(kv_splits=3, merge_mode=2),
                                  dict(kv_splits=3, merge_mode=1), dict(kv_splits=1)])
@pytest.mark.parametrize("paged", [False, True])
def test_graph_replays_match_eager(opts, paged):
    say(f"graph replay paged={paged} {opts}")
    w = synth.small(batch=2, n_q_heads=16, n_kv_heads=4, suffix_len=40, keep=("ratio", 0.2, 0.8))
    dev = Dev(w)
    plan = c2kv.Plan.for_workload(w, **opts).upload()
    ksh, vsh = c2kv.page_shapes(plan)
    kp = torch.empty(ksh, dtype=torch.bfloat16, device="cuda")
    vp = torch.empty(vsh, dtype=torch.bfloat16, device="cuda")

    def run(out, lse):
        if paged:
            c2kv.c2kv_compose(plan, dev.pool, kp, vp)
            c2kv.c2kv_attend(plan, kp, vp, dev.q, dev.k_suf, dev.v_suf, out, lse)
        else:
            c2kv.c2kv_compose_attend(plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out, lse)

    ref, ref_lse = dev.out_like(), dev.lse_like()
    run(ref, ref_lse)
    torch.cuda.synchronize()

    out, lse = dev.out_like(), dev.lse_like()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(out, lse)                      # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(out, lse)
    for i in range(4):
        out.zero_()
        lse.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {i}"
        assert torch.equal(lse, ref_lse), f"replay {i}"
        # eager work of the same plan between replays
        tmp, tmp_lse = dev.out_like(), dev.lse_like()
        run(tmp, tmp_lse)
        torch.cuda.synchronize()
        assert torch.equal(tmp, ref)
