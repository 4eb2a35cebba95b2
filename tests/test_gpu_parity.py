"""GPU parity of the HIP path (through the C ABI) with the float64 oracle.

Every workload runs both ways: c2kv_compose_attend (gather/decode/turn fused
into the attention loads) and c2kv_compose followed by c2kv_attend (paged
cache).  Tolerances are listed in gpu_common.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_17715_amd as c2kv
import synth
from gpu_common import Dev, compare, oracle_ref, run_fused, run_paged, say

pytestmark = pytest.mark.gpu


def _both_paths(w, what, rows=None, **opts):
    ref_out, ref_lse, _ = oracle_ref(w, rows=rows)
    say(f"{what}: fused compose_attend {opts}")
    out, lse, plan, dev = run_fused(w, **opts)
    compare(w, out, lse, ref_out, ref_lse, rows=rows, what=f"{what}/fused")
    say(f"{what}: compose + attend {opts}")
    out2, lse2, _, _, _ = run_paged(w, dev=dev, plan=plan)
    compare(w, out2, lse2, ref_out, ref_lse, rows=rows, what=f"{what}/paged")
    # the two paths round the same values the same way: identical results
    assert torch.equal(out, out2), what
    return plan


# ---------------------------------------------------------------------------
# the five workloads at their full sizes
# ---------------------------------------------------------------------------

def test_tiny_fp32():
    _both_paths(synth.config(1), "tiny-fp32")


def test_llama3_8b_layer_bf16():
    _both_paths(synth.config(2), "llama3-8b-layer")


def test_ragged_batch_bf16():
    _both_paths(synth.config(3), "ragged-batch")


@pytest.mark.parametrize("layer", [0, 31])
def test_int8_layer(layer):
    _both_paths(synth.config(4, layer=layer), f"int8-layer{layer}")


def test_long_suffix_sampled_rows():
    """Full 70B-shaped workload (32768 composed slots, S = 2048) in the launch
    configuration the benchmark times; the oracle computes sampled suffix rows."""
    w = synth.config(5)
    # one suffix token in each of the 64 row blocks of 256 rows (32 tokens of 8
    # heads each), at a different offset in each block so that every in-block
    # position of the causal diagonal tile is met, plus both ends
    G = w.n_q_heads // w.n_kv_heads
    per_block = 256 // G
    rows = sorted({0, 1, w.suffix_len - 1} |
                  {per_block * i + (i % per_block) for i in range(w.suffix_len // per_block)})
    _both_paths(w, "70b-long-suffix", rows=rows)


# ---------------------------------------------------------------------------
# decode steps: one suffix token over the composed cache (split-K over keys)
# ---------------------------------------------------------------------------

def test_decode_small():
    sp = synth.Spec("decode-small", 32, 8, 128, 5e5, "bf16", "bf16", 8, 512, 0, 1, 8,
                    "natural", ("count", 128), 1)
    _both_paths(synth.build(sp, seed=11), "decode-small")


def test_decode_32k_4x():
    _both_paths(synth.config(6), "decode-32k-4x")


def test_decode_128k_4x():
    """The 128k-context decode with 4x compression at full size."""
    _both_paths(synth.config(7), "decode-128k-4x")


@pytest.mark.parametrize("idx", [12, 14, 15])
def test_decode_16k_grid(idx):
    """The 16k-context decode, uncompressed and at 8x and 16x, at full size."""
    _both_paths(synth.config(idx), synth.spec(idx).name)


@pytest.mark.parametrize("head_dim,kv_splits", [(128, 64), (128, 65), (128, 200),
                                                (64, 128), (64, 129), (64, 256)])
def test_merge_many_splits(head_dim, kv_splits):
    """Row blocks of a few rows with many splits are combined one row per
    workgroup, each lane loading a batch of splits (64 at D = 128, 128 at D = 64)
    with the LSEs; counts at, just past and well past one batch take the later
    batches' path.  16384 composed tokens: 256 key tiles per kv-head."""
    sp = synth.Spec("merge-many", 8, 2, head_dim, 5e5, "bf16", "bf16", 4, 4096, 0, 1, 4,
                    "natural", ("all",), 2)
    w = synth.build(sp, seed=23)
    plan = _both_paths(w, f"merge-many D={head_dim} splits={kv_splits}", kv_splits=kv_splits)
    assert plan.info["max_splits"] == kv_splits
    assert plan.info["rows_per_block"] <= 128


@pytest.mark.parametrize("kv_splits", [17, 32, 33, 65])
def test_merge_256_row_blocks_batches(kv_splits):
    """256-row blocks combine their splits in batches of up to 32, loading partial
    rows for the group's own splits only: one batch past the old 16, exactly one
    batch, one split past it, and two batches and a split (4160 composed keys and
    suffix tokens, 65 key tiles per row block)."""
    sp = synth.Spec("merge-256", 8, 2, 128, 5e5, "bf16", "bf16", 4, 1024, 0, 1, 4,
                    "natural", ("all",), 64)
    w = synth.build(sp, seed=29)
    plan = _both_paths(w, f"merge-256 splits={kv_splits}", kv_splits=kv_splits)
    assert plan.info["rows_per_block"] == 256
    assert plan.info["max_splits"] == kv_splits


@pytest.mark.parametrize("suffix_len", [1, 7, 25])
@pytest.mark.parametrize("opts", [dict(kv_splits=1), dict(kv_splits=2), dict(kv_splits=3),
                                  dict(kv_splits=5), dict(kv_splits=3, page_size=128)])
def test_paged_128_row_blocks_tile_counts(suffix_len, opts):
    """128-row blocks over pages keep two tiles in flight in alternating register
    sets, so an item's tile count may be odd or even, and its first and last
    tiles partial; with few suffix tokens most 32-row groups hold no rows."""
    w = synth.small(batch=3, n_q_heads=16, n_kv_heads=4, suffix_len=suffix_len,
                    chunks_per_req=3, keep=("ratio", 0.2, 0.9))
    plan = _both_paths(w, f"paged-128 S={suffix_len} {opts}", rows_per_block=128, **opts)
    assert plan.info["rows_per_block"] == 128


# ---------------------------------------------------------------------------
# keys stored before RoPE; C^2-pattern kept sets at compression 4 / 8 / 10 / 16
# ---------------------------------------------------------------------------

def test_llama3_8b_layer_pre_rope_keys():
    _both_paths(synth.config(10), "llama3-8b-layer-prerope")


def test_llama3_8b_layer_c2_pattern():
    _both_paths(synth.config(11), "llama3-8b-layer-c2x4")


@pytest.mark.parametrize("ratio", [4, 8, 10, 16])
@pytest.mark.parametrize("pre_rope", [False, True])
def test_c2_pattern_ratios(ratio, pre_rope):
    w = synth.small(batch=3, keep=("c2", ratio), n_q_heads=16, n_kv_heads=4, suffix_len=40,
                    chunk_len=300, seed=20 + ratio)
    w = synth.with_overrides(w, keys_pre_rope=pre_rope)
    _both_paths(w, f"c2-pattern-x{ratio}-prerope{int(pre_rope)}")


@pytest.mark.parametrize("pool_dtype", ["f32", "i8"])
def test_pre_rope_other_storage(pool_dtype):
    w = synth.small(pool_dtype=pool_dtype, act_dtype="f32" if pool_dtype == "f32" else "bf16",
                    batch=2, keep=("ratio", 0.2, 0.6), seed=31)
    _both_paths(synth.with_overrides(w, keys_pre_rope=True), f"pre-rope-{pool_dtype}")


# ---------------------------------------------------------------------------
# compose: layout bit-exact, values, delta = 0 copies
# ---------------------------------------------------------------------------

def _check_pages(w, plan, res):
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx, w.seg_new_pos0)
    # layout outputs written by the kernel: bit-exact
    src = res["src"].cpu().numpy()
    pos = res["pos"].cpu().numpy()
    if len(src):
        np.testing.assert_array_equal(src, np.concatenate(lay["src_row"]))
        np.testing.assert_array_equal(pos, np.concatenate(lay["p_new"]))
    np.testing.assert_array_equal(res["bt"].cpu().numpy(), plan.block_table())
    # page contents against the oracle's composed cache
    caches = oracle.compose(lay, w.pool_k, w.pool_v, w.pool_dtype, w.rope_base,
                            w.pool_k_scale, w.pool_v_scale)
    kp = c2kv.to_numpy_f64(res["k_pages"])
    vp = c2kv.to_numpy_f64(res["v_pages"])
    bt = plan.block_table()
    ps = plan.info["page_size"]
    rel = 1e-6 if w.act_dtype == "f32" else 2.0 ** -8
    for b, (kc, vc) in enumerate(caches):
        n = kc.shape[0]
        s = np.arange(n)
        pages = bt[b][s // ps]
        kg = kp[pages, :, s % ps, :]                    # [n, H, D]
        vg = vp[pages, :, :, s % ps]                    # [n, H, D] (pages hold V^T)
        assert np.all(np.abs(kg - kc) <= rel * np.abs(kc) + 1e-6), b
        assert np.all(np.abs(vg - vc) <= rel * np.abs(vc) + 1e-6), b


@pytest.mark.parametrize("pool_dtype", ["f32", "bf16", "i8"])
def test_compose_pages(pool_dtype):
    w = synth.small(pool_dtype=pool_dtype, batch=3, keep=("ratio", 0.05, 0.7))
    for ps in (64, 128):
        say(f"compose pages {pool_dtype} page_size={ps}")
        _, _, plan, _, res = run_paged(w, page_size=ps)
        _check_pages(w, plan, res)


def test_compose_delta0_is_a_bit_exact_copy():
    """With every segment already at its final position (delta = 0), composing
    bf16 keys is a copy: cos = 1 and sin = 0 are exact."""
    w = synth.small(pool_dtype="bf16", batch=2, keep=("ratio", 0.1, 0.9))
    new0 = []
    for r in range(w.batch):
        pos = 0
        for c in range(w.req_seg_off[r], w.req_seg_off[r + 1]):
            new0.append(pos)
            pos += int(w.seg_span[c])
    w = synth.with_overrides(w, seg_orig_pos0=np.array(new0, np.int32))
    _, _, plan, dev, res = run_paged(w)
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx)
    assert all((d == 0).all() for d in lay["delta"])
    kp = res["k_pages"].view(torch.int16).cpu().numpy().view(np.uint16)
    vp = res["v_pages"].view(torch.int16).cpu().numpy().view(np.uint16)
    bt = plan.block_table()
    ps = plan.info["page_size"]
    for b in range(w.batch):
        rows = lay["src_row"][b]
        s = np.arange(len(rows))
        pages = bt[b][s // ps]
        np.testing.assert_array_equal(kp[pages, :, s % ps, :], w.pool_k[rows])
        np.testing.assert_array_equal(vp[pages, :, :, s % ps], w.pool_v[rows])


# ---------------------------------------------------------------------------
# launch shapes: split counts and row blocks do not change the result
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("opts", [dict(kv_splits=1), dict(kv_splits=2), dict(kv_splits=7),
                                  dict(kv_splits=3, merge_mode=1),
                                  dict(kv_splits=3, merge_mode=2),
                                  dict(kv_splits=12, merge_mode=1),
                                  dict(rows_per_block=128), dict(rows_per_block=256),
                                  dict(rows_per_block=256, kv_splits=3, merge_mode=2),
                                  dict(page_size=256)])
def test_launch_shape_invariance(opts):
    w = synth.small(batch=2, n_q_heads=16, n_kv_heads=4, suffix_len=45,
                    keep=("ratio", 0.1, 0.8))
    _both_paths(w, f"shape {opts}", **opts)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def test_single_query_token():
    _both_paths(synth.small(suffix_len=1, batch=2), "S=1")


def test_nothing_kept():
    """No cached slot at all: attention over the causal suffix only."""
    _both_paths(synth.small(keep=("none",), prefix_len=0, batch=2), "nothing kept")


def test_one_cached_token():
    w = synth.small(batch=1, prefix_len=0, chunks_per_req=1, keep=("count", 1), suffix_len=5)
    _both_paths(w, "one cached token")


def test_empty_and_long_requests_in_one_batch():
    w = synth.small(batch=3, prefix_len=0, chunks_per_req=2, keep=("ratio", 0.5, 1.0))
    off = w.seg_kept_off.copy()
    # request 1 keeps nothing: empty its two segments' kept sets
    s0, s1 = w.req_seg_off[1], w.req_seg_off[2]
    kept = np.concatenate([w.kept_idx[off[c]:off[c + 1]] for c in range(w.n_segments)
                           if not (s0 <= c < s1)])
    sizes = [0 if s0 <= c < s1 else off[c + 1] - off[c] for c in range(w.n_segments)]
    w = synth.with_overrides(w, kept_idx=kept.astype(np.int32),
                             seg_kept_off=np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32))
    _both_paths(w, "empty request in batch")


@pytest.mark.parametrize("heads", [(4, 4), (8, 4), (12, 4), (32, 2)])
@pytest.mark.parametrize("rows_per_block", [64, 128, 256])
def test_gqa_group_sizes(heads, rows_per_block):
    """Query heads per kv-head G = 1, 2, 3 and 16: a row block's rows r = t*G + (h mod G)
    then start and end at any head of a token."""
    hq, hkv = heads
    w = synth.small(batch=2, n_q_heads=hq, n_kv_heads=hkv, suffix_len=37,
                    keep=("ratio", 0.2, 0.8), seed=40 + hq)
    _both_paths(w, f"G={hq // hkv} rows={rows_per_block}", rows_per_block=rows_per_block)


def test_head_dim_64_bf16_and_int8():
    for dt in ("bf16", "i8"):
        _both_paths(synth.small(pool_dtype=dt, head_dim=64, batch=2), f"d=64 {dt}")


def test_head_dim_128_fp32():
    _both_paths(synth.small(pool_dtype="f32", head_dim=128, batch=2), "fp32 d=128")


def test_repeated_chunks_and_explicit_placement():
    w = synth.small(batch=1, chunks_per_req=3, n_pool_chunks=3, prefix_len=0, suffix_len=20)
    w = synth.with_overrides(
        w, req_seg_off=np.array([0, 3], np.int32), seg_row0=np.array([0, 200, 0], np.int64),
        seg_span=np.array([200, 200, 200], np.int32),
        seg_orig_pos0=np.array([0, 0, 7], np.int32),
        seg_new_pos0=np.array([1000, 50, 5000], np.int32),
        seg_kept_off=np.array([0, 70, 75, 145], np.int32),
        kept_idx=np.concatenate([np.arange(0, 140, 2), np.arange(5), np.arange(0, 140, 2)]
                                ).astype(np.int32))
    _both_paths(w, "repeated chunk, explicit placement")


def test_explicit_placement_golden():
    """The hand-worked explicit-placement layout (out of order, overlapping, a
    segment that keeps nothing, negative deltas; the furthest span is not the
    last segment's), end to end through both paths against the oracle."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                    "layout_explicit_placement.json")))
    w = synth.small(batch=2, suffix_len=19)
    a = lambda k, t: np.array(g[k], t)
    w = synth.with_overrides(
        w, req_seg_off=a("req_seg_off", np.int32), seg_row0=a("seg_row0", np.int64),
        seg_span=a("seg_span", np.int32), seg_orig_pos0=a("seg_orig_pos0", np.int32),
        seg_new_pos0=a("seg_new_pos0", np.int32), seg_kept_off=a("seg_kept_off", np.int32),
        kept_idx=a("kept_idx", np.int32))
    plan = _both_paths(w, "explicit placement golden")
    n, e = plan.requests()
    assert list(e) == g["expect"]["span_end"]


def test_gqa_groups():
    for hq, hkv in [(8, 8), (16, 2), (12, 4)]:
        _both_paths(synth.small(n_q_heads=hq, n_kv_heads=hkv, batch=1), f"Hq={hq} Hkv={hkv}")


def test_lse_optional_and_plan_reuse_across_layers():
    """One plan serves several layers (the kept set is layer-independent); lse may be NULL."""
    sp = synth.spec(4)
    sp = synth.Spec(**{**sp.__dict__, "n_pool_chunks": 8, "chunks_per_req": 8})
    ws = [synth.build(sp, layer=l, seed=7) for l in range(3)]
    plan = c2kv.Plan.for_workload(ws[0]).upload()
    for l, w in enumerate(ws):
        dev = Dev(w)
        out = dev.out_like()
        c2kv.c2kv_compose_attend(plan, dev.pool, dev.q, dev.k_suf, dev.v_suf, out, None)
        torch.cuda.synchronize()
        ref_out, ref_lse, _ = oracle_ref(w)
        lse = torch.from_numpy(ref_lse.astype(np.float32))
        compare(w, out, lse, ref_out, ref_lse, what=f"layer {l}")


@pytest.mark.parametrize("pool_dtype", ["bf16", "i8", "f32"])
def test_pool_rows_past_4gib(pool_dtype):
    """Kept rows more than 4.5 GiB into the pool: the same rows moved r0 rows up
    in a larger pool (seg_row0 shifted by r0) give bit-identical outputs, pages
    and source rows on both paths, and the unshifted run meets the oracle."""
    w = synth.small(pool_dtype=pool_dtype, n_q_heads=16, n_kv_heads=8, suffix_len=21)
    n, H, D = w.pool_k.shape
    esz = {"bf16": 2, "i8": 1, "f32": 4}[pool_dtype]
    r0 = -(-(9 << 29) // (H * D * esz))
    say(f"pool past 4.5 GiB {pool_dtype}: r0 = {r0} rows, {(r0 + n) * H * D * esz / 2**30:.2f} GiB")
    ref_out, ref_lse, _ = oracle_ref(w)
    out, lse, plan, dev = run_fused(w)
    compare(w, out, lse, ref_out, ref_lse, what="pool4g/base")
    out_p, lse_p, _, _, pg = run_paged(w, dev=dev, plan=plan)
    assert torch.equal(out_p, out)

    def moved(t):
        big = torch.zeros((r0 + t.shape[0],) + tuple(t.shape[1:]), dtype=t.dtype, device="cuda")
        big[r0:] = t
        return big

    # the descriptor holds raw pointers: keep the moved tensors referenced
    held = [moved(dev.k), moved(dev.v), None if dev.ks is None else moved(dev.ks),
            None if dev.vs is None else moved(dev.vs)]
    dev.pool = c2kv.pool_desc(*held)
    w2 = synth.with_overrides(w, seg_row0=(w.seg_row0 + r0).astype(w.seg_row0.dtype))
    out2, lse2, plan2, _ = run_fused(w2, dev=dev)
    assert torch.equal(out2, out) and torch.equal(lse2, lse)
    out3, lse3, _, _, pg2 = run_paged(w2, dev=dev, plan=plan2)
    assert torch.equal(out3, out) and torch.equal(lse3, lse_p)
    assert torch.equal(pg2["k_pages"], pg["k_pages"]) and torch.equal(pg2["v_pages"], pg["v_pages"])
    assert torch.equal(pg2["src"], pg["src"] + r0)
    dev.pool = None
    del held
    torch.cuda.empty_cache()


def _replicate(w, B):
    """B identical requests: every request repeats the segments, kept sets and
    suffix inputs of request 0 of w (a one-request workload); the pool is shared."""
    kept_counts = np.diff(w.seg_kept_off)
    tile = lambda a: np.tile(a, (B,) + (1,) * (a.ndim - 1))
    return synth.with_overrides(
        w, req_seg_off=(np.arange(B + 1) * w.n_segments).astype(w.req_seg_off.dtype),
        seg_row0=tile(w.seg_row0), seg_span=tile(w.seg_span),
        seg_orig_pos0=tile(w.seg_orig_pos0),
        seg_new_pos0=None if w.seg_new_pos0 is None else tile(w.seg_new_pos0),
        seg_kept_off=np.concatenate([[0], np.cumsum(tile(kept_counts))]).astype(
            w.seg_kept_off.dtype),
        kept_idx=tile(w.kept_idx), q=tile(w.q), k_suf=tile(w.k_suf), v_suf=tile(w.v_suf))


def test_pages_past_4gib():
    """Composed pages more than 4 GiB into k_pages and v_pages: 36 copies of one
    64k-token decode request, with the same key splits, each give the output of
    the request alone bit for bit, and that output meets the oracle."""
    sp = synth.Spec("decode-64k-pages", 32, 8, 128, 5e5, "bf16", "bf16", 8, 8192, 0, 1, 8,
                    "natural", ("all",), 1)
    w = synth.build(sp, seed=23)
    assert w.batch == 1
    ref_out, ref_lse, _ = oracle_ref(w)
    say("pages past 4 GiB: one request")
    out, lse, _, _, _ = run_paged(w, kv_splits=4)
    compare(w, out, lse, ref_out, ref_lse, what="pages4g/one")
    B = 36
    wB = _replicate(w, B)
    plan = c2kv.Plan.for_workload(wB, kv_splits=4).upload()
    page_bytes = plan.info["n_pages"] * w.n_kv_heads * plan.info["page_size"] * w.head_dim * 2
    say(f"pages past 4 GiB: {B} requests, k_pages {page_bytes / 2**30:.2f} GiB")
    assert page_bytes > (4 << 30)
    outB, lseB, _, _, pg = run_paged(wB, plan=plan)
    for b in range(B):
        assert torch.equal(outB[b], out[0]), b
        assert torch.equal(lseB[b], lse[0]), b
    # the last request's pages (past 4 GiB) hold what the first request's hold
    bt = pg["bt"].cpu().numpy()
    npg = plan.info["max_pages"]
    assert (bt[B - 1] == bt[B - 1][0] + np.arange(npg)).all() and bt[0][0] == 0
    last = slice(int(bt[B - 1][0]), int(bt[B - 1][0]) + npg)
    assert torch.equal(pg["k_pages"][last], pg["k_pages"][:npg])
    assert torch.equal(pg["v_pages"][last], pg["v_pages"][:npg])
    del pg
    torch.cuda.empty_cache()
