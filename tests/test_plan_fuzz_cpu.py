"""Seeded random segment descriptors through the host plan (CPU): the composed
slot table (source row, new position, delta), composed lengths and span ends
equal the oracle's layout bit for bit, and the block table covers exactly the
composed slots.  Draws include empty kept sets, single-token spans, repeated
chunks, explicit and accumulated placements, overlapping placements, the
compressed pool layout and both key encodings."""
import numpy as np
import pytest

import oracle
import paper_2607_17715_amd as c2kv


def _descriptor(r):
    B = int(r.integers(1, 5))
    n_pool_rows = 4000
    req_seg_off = [0]
    seg_row0, seg_span, seg_orig, kept_off, kept = [], [], [], [0], []
    for _ in range(B):
        for _ in range(int(r.integers(0, 5))):
            span = int(r.choice([1, 2, 7, 63, 64, 65, 200]))
            row0 = int(r.integers(0, n_pool_rows - span))
            m = int(r.integers(0, span + 1)) if r.integers(3) else span
            idx = np.sort(r.choice(span, size=m, replace=False)).astype(np.int32)
            seg_row0.append(row0)
            seg_span.append(span)
            seg_orig.append(int(r.integers(0, 5000)))
            kept.append(idx)
            kept_off.append(kept_off[-1] + m)
        req_seg_off.append(len(seg_row0))
    n_seg = len(seg_row0)
    new0 = None
    if r.integers(2) and n_seg:
        new0 = r.integers(0, 20000, size=n_seg).astype(np.int32)
    return dict(req_seg_off=np.array(req_seg_off, np.int32),
                seg_row0=np.array(seg_row0, np.int64), seg_span=np.array(seg_span, np.int32),
                seg_orig_pos0=np.array(seg_orig, np.int32),
                seg_kept_off=np.array(kept_off, np.int32),
                kept_idx=np.concatenate(kept) if kept else np.zeros(0, np.int32),
                seg_new_pos0=new0)


@pytest.mark.parametrize("i", range(200))
def test_random_descriptor_layout(i):
    r = np.random.default_rng(5100 + i)
    d = _descriptor(r)
    compressed = bool(r.integers(4) == 0)
    pre_rope = bool(r.integers(4) == 0)
    if compressed:
        # the k-th kept token of a segment lives in row seg_row0 + k
        d["seg_row0"] = np.cumsum(np.concatenate([[0], np.diff(d["seg_kept_off"])]))[:-1].astype(np.int64)
    ps = int(r.choice([64, 128, 256]))
    plan = c2kv.Plan(8, 2, 128, "bf16", 5e5, d["req_seg_off"], d["seg_row0"], d["seg_span"],
                     d["seg_orig_pos0"], d["seg_kept_off"], d["kept_idx"], int(r.integers(1, 70)),
                     seg_new_pos0=d["seg_new_pos0"], keys_pre_rope=pre_rope,
                     pool_compressed=compressed, page_size=ps)
    lay = oracle.compose_layout(d["req_seg_off"], d["seg_row0"], d["seg_span"],
                                d["seg_orig_pos0"], d["seg_kept_off"], d["kept_idx"],
                                d["seg_new_pos0"], compressed=compressed)
    n, e = plan.requests()
    np.testing.assert_array_equal(n, lay["composed_len"])
    np.testing.assert_array_equal(e, lay["span_end"])
    src, pos, dl = plan.slots()
    cat = lambda xs: np.concatenate(xs) if len(xs) and sum(len(x) for x in xs) else np.zeros(0)
    np.testing.assert_array_equal(src, cat(lay["src_row"]))
    np.testing.assert_array_equal(pos, cat(lay["p_new"]))
    np.testing.assert_array_equal(dl, cat(lay["delta"]))
    bt = plan.block_table()
    used = []
    for b in range(len(n)):
        need = -(-int(n[b]) // ps)
        assert all(bt[b][:need] >= 0) and all(bt[b][need:] == -1)
        used += list(bt[b][:need])
    assert sorted(used) == list(range(plan.info["n_pages"]))
