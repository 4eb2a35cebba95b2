"""The load step (Appendix C): chunks stored compressed, pools in page-locked
host memory read in place by the kernels, and copies of the rows a plan reads
into a device pool (c2kv_load).  Every path must give the same bits as the
device pool of whole chunks, and match the oracle."""
import numpy as np
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, compare, oracle_ref, run_fused, run_paged, say

pytestmark = pytest.mark.gpu


def _fused_from(plan, pool, dev):
    out, lse = dev.out_like(), dev.lse_like()
    c2kv.c2kv_compose_attend(plan, pool, dev.q, dev.k_suf, dev.v_suf, out, lse)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("idx", [2, 3, 4])
def test_compressed_pool_equals_whole_chunks(idx):
    w = synth.config(idx)
    wc = synth.compress_pool(w)
    say(f"compressed pool, workload {idx}: {w.pool_k.shape[0]} -> {wc.pool_k.shape[0]} rows")
    ref, ref_lse, _ = oracle_ref(wc)
    out, lse, _, _ = run_fused(w)
    outc, lsec, plan, dev = run_fused(wc)
    compare(wc, outc, lsec, ref, ref_lse, what=f"compressed-{idx}/fused")
    assert torch.equal(out, outc) and torch.equal(lse, lsec)
    outp, lsep, _, _, _ = run_paged(wc, dev=dev, plan=plan)
    assert torch.equal(outp, outc)


@pytest.mark.parametrize("idx", [2, 4])
def test_host_pool_read_in_place(idx):
    """Kernels read a pool in page-locked host memory over the host link."""
    wc = synth.compress_pool(synth.config(idx))
    out, lse, plan, dev = run_fused(wc)
    host = c2kv.HostPool(wc.pool_k, wc.pool_v, wc.pool_dtype, wc.pool_k_scale, wc.pool_v_scale)
    say(f"host pool, workload {idx}: {host.nbytes / 1e6:.1f} MB")
    outh, lseh = _fused_from(plan, host.desc, dev)
    assert torch.equal(out, outh) and torch.equal(lse, lseh)
    # the paged path reads the host pool too
    ks, vs = c2kv.page_shapes(plan)
    act = torch.bfloat16
    kp = torch.empty(ks, dtype=act, device="cuda")
    vp = torch.empty(vs, dtype=act, device="cuda")
    c2kv.c2kv_compose(plan, host.desc, kp, vp)
    outp = dev.out_like()
    c2kv.c2kv_attend(plan, kp, vp, dev.q, dev.k_suf, dev.v_suf, outp, None)
    torch.cuda.synchronize()
    assert torch.equal(out, outp)
    host.close()


@pytest.mark.parametrize("compressed", [True, False])
@pytest.mark.parametrize("idx", [2, 4])
def test_load_copies_exactly_the_rows_a_plan_reads(idx, compressed):
    w = synth.config(idx)
    if compressed:
        w = synth.compress_pool(w)
    out, lse, plan, dev = run_fused(w)
    host = c2kv.HostPool(w.pool_k, w.pool_v, w.pool_dtype, w.pool_k_scale, w.pool_v_scale)
    # a device pool of the same shape, filled with a marker value first
    dk, dv = torch.full_like(dev.k, 7), torch.full_like(dev.v, 7)
    dks = None if dev.ks is None else torch.full_like(dev.ks, -3.0)
    dvs = None if dev.vs is None else torch.full_like(dev.vs, -3.0)
    dst = c2kv.pool_desc(dk, dv, dks, dvs)
    c2kv.c2kv_load(plan, host.desc, dst)
    torch.cuda.synchronize()
    src_rows = np.unique(plan.slots()[0])
    read = np.zeros(w.pool_k.shape[0], bool)
    read[src_rows] = True
    # rows the plan reads are copies of the source; copied ranges run first to
    # last kept row of each segment, and no row outside them is touched
    bits = torch.int8 if w.pool_dtype == "i8" else torch.int16
    marker = torch.full((1,), 7, dtype=dk.dtype).view(bits).item()
    got_k = dk.view(bits).cpu().numpy()
    ref_k = np.ascontiguousarray(w.pool_k).view(np.int8 if w.pool_dtype == "i8" else np.int16)
    np.testing.assert_array_equal(got_k[read], ref_k[read])
    touched = (got_k != marker).reshape(len(read), -1).any(axis=1) | read
    if compressed:
        assert touched.all()
    say(f"load idx {idx} compressed {compressed}: {int(read.sum())} rows read, "
        f"{int(touched.sum())} rows copied of {len(read)}")
    outl, lsel = _fused_from(plan, dst, dev)
    assert torch.equal(out, outl) and torch.equal(lse, lsel)
    host.close()
