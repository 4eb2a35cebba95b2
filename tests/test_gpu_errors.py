"""The C ABI's call-time checks on the GPU: with an uploaded plan, each
documented rejection returns its status and a message, and launches nothing
(outputs, pages and the plan keep working as before).  Rejected descriptors are
checked before any pointer in them is used."""
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, run_fused, say

pytestmark = pytest.mark.gpu


def _rejected(fn):
    with pytest.raises(c2kv.C2KVError) as ei:
        fn()
    return ei.value.status, str(ei.value)


def test_call_time_rejections_launch_nothing():
    say("call-time rejections")
    w = synth.small(batch=2)
    ref_out, ref_lse, plan, dev = run_fused(w)
    mx = plan.info["max_src_row"]
    n = dev.k.shape[0]
    assert mx == n - 1 or mx < n
    ksh, vsh = c2kv.page_shapes(plan)
    kp = torch.full(ksh, 3.0, dtype=torch.bfloat16, device="cuda")
    vp = torch.full(vsh, 3.0, dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(dev.q, 7.0)
    lse = torch.full_like(ref_lse, 7.0)
    k, v = dev.k.data_ptr(), dev.v.data_ptr()
    i8k = torch.zeros(dev.k.shape, dtype=torch.int8, device="cuda")
    i8v = torch.zeros(dev.v.shape, dtype=torch.int8, device="cuda")
    sc = torch.ones(dev.k.shape[:2], dtype=torch.float32, device="cuda")
    i8pool = c2kv.pool_desc(i8k, i8v, sc, sc)
    short = c2kv.pool_desc(dev.k[:mx], dev.v[:mx])
    E = c2kv
    fused = lambda pool, q=dev.q, o=out: c2kv.c2kv_compose_attend(
        plan, pool, q, dev.k_suf, dev.v_suf, o, lse)
    paged = lambda a, b, o=out: c2kv.c2kv_attend(plan, a, b, dev.q, dev.k_suf, dev.v_suf, o, lse)
    cases = [
        ("pool shorter than the rows read", lambda: fused(short), E.C2KV_E_INVAL, "pool row"),
        ("compose from a short pool", lambda: c2kv.c2kv_compose(plan, short, kp, vp),
         E.C2KV_E_INVAL, "pool row"),
        ("NULL q", lambda: fused(dev.pool, q=None), E.C2KV_E_INVAL, "NULL"),
        ("NULL out", lambda: fused(dev.pool, o=None), E.C2KV_E_INVAL, "NULL"),
        ("NULL out (paged)", lambda: paged(kp, vp, o=None), E.C2KV_E_INVAL, "NULL"),
        ("NULL k_pages", lambda: paged(None, vp), E.C2KV_E_INVAL, "k_pages"),
        ("NULL v_pages (compose)", lambda: c2kv.c2kv_compose(plan, dev.pool, kp, None),
         E.C2KV_E_INVAL, "k_pages"),
        ("NULL pool K", lambda: fused(c2kv.PoolDesc(c2kv.C2KV_BF16, None, v, None, None, n)),
         E.C2KV_E_INVAL, "NULL"),
        ("unknown pool dtype", lambda: fused(c2kv.PoolDesc(9, k, v, None, None, n)),
         E.C2KV_E_INVAL, "dtype"),
        ("f32 pool under bf16 activations",
         lambda: fused(c2kv.PoolDesc(c2kv.C2KV_F32, k, v, None, None, n)),
         E.C2KV_E_UNSUPPORTED, "combination"),
        ("int8 pool without scales",
         lambda: fused(c2kv.PoolDesc(c2kv.C2KV_I8, i8k.data_ptr(), i8v.data_ptr(), None, None, n)),
         E.C2KV_E_INVAL, "scale"),
        ("load between pools of two dtypes", lambda: c2kv.c2kv_load(plan, dev.pool, i8pool),
         E.C2KV_E_INVAL, "dtype"),
    ]
    for name, fn, want, text in cases:
        st, msg = _rejected(fn)
        say(f"{name}: {msg}")
        assert st == want and text in msg, (name, st, msg)
    torch.cuda.synchronize()
    assert (out == 7.0).all() and (lse == 7.0).all()
    assert (kp == 3.0).all() and (vp == 3.0).all()
    # a pool of exactly the rows read is enough, and the plan still gives its result
    exact = c2kv.pool_desc(dev.k[:mx + 1], dev.v[:mx + 1])
    fused(exact)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
