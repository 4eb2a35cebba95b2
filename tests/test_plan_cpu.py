"""Host side of the C ABI, on the CPU: the library loads and exports every call
include/c2kv.h declares; the plan's kept-token layout equals the oracle's
bit for bit; bad descriptors are rejected with the documented status codes."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import oracle
import paper_2607_17715_amd as c2kv
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "c2kv.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    declared = set(re.findall(r"\b(c2kv_[a-z_]+)\s*\(", hdr))
    assert {"c2kv_compose", "c2kv_attend", "c2kv_compose_attend"} <= declared
    lib = ctypes.CDLL(c2kv.LIB_PATH)
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared == set(c2kv.EXPORTED)


def _oracle_layout(w):
    return oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                 w.seg_kept_off, w.kept_idx, w.seg_new_pos0)


def _assert_layout_equal(w, plan):
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx, w.seg_new_pos0,
                                compressed=w.pool_compressed)
    n, e = plan.requests()
    assert list(n) == list(map(int, lay["composed_len"]))
    assert list(e) == list(map(int, lay["span_end"]))
    src, pos, dl = plan.slots()
    np.testing.assert_array_equal(src, np.concatenate(lay["src_row"]) if len(src) else src)
    np.testing.assert_array_equal(pos, np.concatenate(lay["p_new"]) if len(pos) else pos)
    np.testing.assert_array_equal(dl, np.concatenate(lay["delta"]) if len(dl) else dl)


@pytest.mark.parametrize("idx", [1, 2, 4, 5, 6, 10, 11, 13, 18])
def test_layout_bit_exact_configs(idx):
    w = synth.config(idx)
    _assert_layout_equal(w, c2kv.Plan.for_workload(w))


@pytest.mark.parametrize("idx", [1, 2, 3, 4])
def test_layout_bit_exact_compressed_pools(idx):
    w = synth.compress_pool(synth.config(idx))
    plan = c2kv.Plan.for_workload(w)
    _assert_layout_equal(w, plan)
    assert plan.info["max_src_row"] == w.pool_k.shape[0] - 1


def test_layout_bit_exact_ragged_and_edges():
    for kw in [dict(keep=("ratio", 0.0, 0.4), batch=4, chunks_per_req=5, prefix_len=0),
               dict(keep=("c2", 4), batch=2),
               dict(keep=("none",), batch=2, prefix_len=3),
               dict(keep=("all",), batch=1, chunk_len=65)]:
        w = synth.small(**kw)
        _assert_layout_equal(w, c2kv.Plan.for_workload(w))


def test_layout_explicit_placement_and_repeats():
    w = synth.small(batch=1, chunks_per_req=3, n_pool_chunks=3, prefix_len=0)
    # place the same chunk twice, with a gap, and one segment before another's span end
    w = synth.with_overrides(
        w, req_seg_off=np.array([0, 3], np.int32), seg_row0=np.array([0, 200, 0], np.int64),
        seg_span=np.array([200, 200, 200], np.int32),
        seg_orig_pos0=np.array([0, 0, 7], np.int32),
        seg_new_pos0=np.array([1000, 50, 5000], np.int32),
        seg_kept_off=np.array([0, 3, 5, 8], np.int32),
        kept_idx=np.array([0, 10, 199, 3, 4, 0, 10, 199], np.int32))
    plan = c2kv.Plan.for_workload(w)
    _assert_layout_equal(w, plan)
    n, e = plan.requests()
    assert e[0] == 5200


def _golden_workload(name):
    """A small workload whose layout is the hand-worked golden `name` (pool values
    from the seeded generator; the golden's rows all lie inside its pool)."""
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", name)))
    w = synth.small(batch=len(g["req_seg_off"]) - 1, suffix_len=19)
    a = lambda k, t: None if g.get(k) is None else np.array(g[k], t)
    return g, synth.with_overrides(
        w, req_seg_off=a("req_seg_off", np.int32), seg_row0=a("seg_row0", np.int64),
        seg_span=a("seg_span", np.int32), seg_orig_pos0=a("seg_orig_pos0", np.int32),
        seg_new_pos0=a("seg_new_pos0", np.int32), seg_kept_off=a("seg_kept_off", np.int32),
        kept_idx=a("kept_idx", np.int32))


@pytest.mark.parametrize("name", ["layout_worked_example.json", "layout_explicit_placement.json"])
def test_plan_layout_matches_hand_worked_golden(name):
    """The plan builder's slot table and span ends against the values worked by
    hand (the explicit-placement golden has its furthest span on a segment that
    is not the last)."""
    g, w = _golden_workload(name)
    plan = c2kv.Plan.for_workload(w)
    n, e = plan.requests()
    assert list(n) == g["expect"]["composed_len"]
    assert list(e) == g["expect"]["span_end"]
    src, pos, dl = plan.slots()
    assert list(src) == [x for r in g["expect"]["src_row"] for x in r]
    assert list(pos) == [x for r in g["expect"]["p_new"] for x in r]
    assert list(dl) == [x for r in g["expect"]["delta"] for x in r]


def test_zero_span_is_rejected():
    w = synth.small(batch=1, chunks_per_req=2, prefix_len=0)
    span = w.seg_span.copy()
    span[1] = 0
    kept_off = w.seg_kept_off.copy()
    kept_off[2] = kept_off[1]
    w = synth.with_overrides(w, seg_span=span, seg_kept_off=kept_off,
                             kept_idx=w.kept_idx[:kept_off[1]])
    with pytest.raises(c2kv.C2KVError) as ei:
        c2kv.Plan.for_workload(w)
    assert ei.value.status == c2kv.C2KV_E_INVAL and "seg_span" in str(ei.value)


def test_static_entry_rejects_plans_beyond_its_array():
    """c2kv_compose_attend_static refuses a plan whose tables and partials exceed
    the static array, before any device work (so this runs without a GPU)."""
    w = synth.small(batch=4, n_q_heads=32, n_kv_heads=8, suffix_len=64, keep=("all",),
                    chunk_len=1000, chunks_per_req=5)
    plan = c2kv.Plan.for_workload(w, kv_splits=64, rows_per_block=256)
    assert plan.info["workspace_bytes"] > c2kv.STATIC_SCRATCH_BYTES
    pool = c2kv.PoolDesc(c2kv.C2KV_BF16, 16, 16, None, None, 1 << 20)
    st = c2kv.lib().c2kv_compose_attend_static(plan.handle, ctypes.byref(pool), 16, 16, 16, 16,
                                               None, None)
    assert st == c2kv.C2KV_E_WORKSPACE
    assert b"static" in c2kv.lib().c2kv_last_error()


def test_block_table_pages():
    w = synth.small(batch=3, keep=("ratio", 0.2, 0.9))
    for ps in (64, 128, 256):
        plan = c2kv.Plan.for_workload(w, page_size=ps)
        n, _ = plan.requests()
        bt = plan.block_table()
        used = []
        for b in range(len(n)):
            need = -(-int(n[b]) // ps)
            row = bt[b]
            assert all(row[:need] >= 0) and all(row[need:] == -1)
            used += list(row[:need])
        assert sorted(used) == list(range(plan.info["n_pages"]))


def test_workspace_and_work_list_sizes():
    for idx in (1, 2, 4, 5):
        w = synth.config(idx)
        plan = c2kv.Plan.for_workload(w)
        i = plan.info
        assert i["workspace_bytes"] > 0 and i["workspace_bytes"] % 256 == 0
        assert i["n_work_items"] >= i["n_merge_groups"]
        assert i["rows_per_block"] in (64, 128, 256)
    # forced split count is honoured
    w = synth.config(2)
    assert c2kv.Plan.for_workload(w, kv_splits=1).info["n_merge_groups"] == 0
    assert c2kv.Plan.for_workload(w, kv_splits=3).info["max_splits"] == 3


def _expect_status(status, fn):
    with pytest.raises(c2kv.C2KVError) as ei:
        fn()
    assert ei.value.status == status, str(ei.value)


def test_validation_errors():
    w = synth.small(batch=1)

    def mk(**kw):
        args = dict(n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                    act_dtype=w.act_dtype, rope_base=w.rope_base, req_seg_off=w.req_seg_off,
                    seg_row0=w.seg_row0, seg_span=w.seg_span, seg_orig_pos0=w.seg_orig_pos0,
                    seg_kept_off=w.seg_kept_off, kept_idx=w.kept_idx, suffix_len=w.suffix_len)
        args.update(kw)
        return lambda: c2kv.Plan(**args)

    mk()()  # the baseline is valid
    E = c2kv
    _expect_status(E.C2KV_E_INVAL, mk(n_q_heads=7))
    _expect_status(E.C2KV_E_UNSUPPORTED, mk(head_dim=96))
    _expect_status(E.C2KV_E_INVAL, mk(head_dim=63))
    _expect_status(E.C2KV_E_INVAL, mk(suffix_len=0))
    _expect_status(E.C2KV_E_INVAL, mk(rope_base=-1.0))
    _expect_status(E.C2KV_E_INVAL, mk(page_size=100))
    _expect_status(E.C2KV_E_INVAL, mk(rows_per_block=48))
    _expect_status(E.C2KV_E_INVAL, mk(rows_per_block=96))
    mk(rows_per_block=64)()                                         # 64-row blocks are valid
    _expect_status(E.C2KV_E_INVAL, mk(merge_mode=3))
    mk(keys_pre_rope=True)()                                        # the other key encoding
    bad = w.kept_idx.copy()
    bad[0], bad[1] = bad[1], bad[0]
    _expect_status(E.C2KV_E_INVAL, mk(kept_idx=bad))                  # not ascending
    bad = w.kept_idx.copy()
    bad[w.seg_kept_off[1] - 1] = w.seg_span[0]
    _expect_status(E.C2KV_E_INVAL, mk(kept_idx=bad))                  # outside the span
    row0 = w.seg_row0.copy()
    row0[0] = -5
    _expect_status(E.C2KV_E_INVAL, mk(seg_row0=row0))
    off = w.req_seg_off.copy()
    off[-1] += 1
    _expect_status(E.C2KV_E_INVAL, mk(req_seg_off=off))
    _expect_status(E.C2KV_E_INVAL,
                   mk(seg_new_pos0=np.full(len(w.seg_row0), 2**31 - 10, np.int32)))
    row0 = w.seg_row0.copy()
    row0[-1] = 2**31
    _expect_status(E.C2KV_E_UNSUPPORTED, mk(seg_row0=row0))


def test_key_encoding_and_pool_layout_are_validated():
    w = synth.small(batch=1)
    a = {k: np.ascontiguousarray(getattr(w, k)) for k in
         ("req_seg_off", "seg_row0", "seg_span", "seg_orig_pos0", "seg_kept_off", "kept_idx")}
    cfg = c2kv.AttnCfg(w.n_q_heads, w.n_kv_heads, w.head_dim, c2kv.C2KV_BF16, w.rope_base, 0.0)
    ptr = lambda x: x.ctypes.data_as(ctypes.c_void_p)
    for enc, lay, want in ((c2kv.C2KV_KEYS_ROPE_AT_ORIG, 0, c2kv.C2KV_OK),
                           (c2kv.C2KV_KEYS_PRE_ROPE, 0, c2kv.C2KV_OK),
                           (0, c2kv.C2KV_POOL_COMPRESSED, c2kv.C2KV_OK),
                           (2, 0, c2kv.C2KV_E_INVAL), (-1, 0, c2kv.C2KV_E_INVAL),
                           (0, 2, c2kv.C2KV_E_INVAL), (0, -1, c2kv.C2KV_E_INVAL)):
        desc = c2kv.ComposeDesc(w.batch, w.n_segments, ptr(a["req_seg_off"]), ptr(a["seg_row0"]),
                                ptr(a["seg_span"]), ptr(a["seg_orig_pos0"]), None,
                                ptr(a["seg_kept_off"]), ptr(a["kept_idx"]), enc, lay)
        h = ctypes.c_void_p()
        st = c2kv.lib().c2kv_plan_create(ctypes.byref(cfg), ctypes.byref(desc), w.suffix_len,
                                         None, ctypes.byref(h))
        assert st == want, (enc, st)
        if st == c2kv.C2KV_OK:
            c2kv.lib().c2kv_plan_destroy(h)


def test_calls_need_an_uploaded_plan():
    w = synth.small(batch=1)
    plan = c2kv.Plan.for_workload(w)
    lib = c2kv.lib()
    st = lib.c2kv_attend(plan.handle, None, None, None, None, None, None, None, None)
    assert st == c2kv.C2KV_E_STATE
    assert b"upload" in lib.c2kv_last_error()
    st = lib.c2kv_plan_upload(plan.handle, None, 0, None)
    assert st == c2kv.C2KV_E_WORKSPACE
    st = lib.c2kv_plan_upload(plan.handle, ctypes.c_void_p(256), 16, None)
    assert st == c2kv.C2KV_E_WORKSPACE                              # too small
    st = lib.c2kv_plan_upload(plan.handle, ctypes.c_void_p(100), 1 << 40, None)
    assert st == c2kv.C2KV_E_WORKSPACE                              # misaligned


def test_sif_row_blocks_need_no_merge():
    """A SIF row block that sees several key ranges (sink, own block, original
    tokens) is one work item running through them: with a row block per CU and
    more, nothing is split or merged; forced splits still merge."""
    w = synth.sif(batch=4, n_tokens=512, block=4, sink=4, n_q_heads=32, n_kv_heads=8, seed=950)
    for rb in (64, 128, 256):
        i = c2kv.Plan.for_sif(w, rows_per_block=rb).info
        assert i["n_merge_groups"] == 0 and i["max_splits"] == 1, (rb, i)
    i = c2kv.Plan.for_sif(w, kv_splits=2).info
    assert i["n_merge_groups"] > 0 and i["max_splits"] >= 2


def test_binding_refuses_to_import_without_the_library(tmp_path):
    """No fallback: with the library missing, importing the binding raises."""
    import subprocess
    import sys
    env = dict(os.environ, C2KV_LIBRARY=str(tmp_path / "missing" / "libc2kv.so"))
    r = subprocess.run([sys.executable, "-c", "import paper_2607_17715_amd"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "is not built" in r.stderr
