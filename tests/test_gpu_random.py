"""A seeded sweep of small random configurations through both HIP paths
(fused compose_attend, and compose + attend over pages) against the float64
oracle: storage and activation dtypes, head sizes, GQA group sizes, suffix
lengths, kept-set patterns, key encodings, compressed pools and launch shapes
drawn together, so that combinations the targeted tests do not name are
covered too.  Every case is printed before it runs."""
import numpy as np
import pytest
import torch

import paper_2607_17715_amd as c2kv
import synth
from gpu_common import compare, oracle_ref, run_fused, run_paged, say

pytestmark = pytest.mark.gpu

N_CASES = 64


def _case(i):
    r = np.random.default_rng(7700 + i)
    pool_dtype = ["f32", "bf16", "i8"][r.integers(3)]
    hq, hkv = [(4, 4), (8, 2), (12, 4), (16, 4), (8, 1)][r.integers(5)]
    keep = [("ratio", 0.05, 0.9), ("c2", int(r.choice([4, 8, 16]))),
            ("count", int(r.integers(1, 60))), ("all",), ("ratio", 0.3, 0.3)][r.integers(5)]
    w = synth.small(pool_dtype=pool_dtype, n_q_heads=hq, n_kv_heads=hkv,
                    head_dim=int(r.choice([64, 128])), batch=int(r.integers(1, 4)),
                    chunks_per_req=int(r.integers(1, 4)), n_pool_chunks=5,
                    chunk_len=int(r.choice([65, 130, 200])), prefix_len=int(r.choice([0, 13])),
                    suffix_len=int(r.choice([1, 5, 33, 64, 100])), keep=keep, seed=8800 + i)
    if r.integers(4) == 0:
        w = synth.with_overrides(w, keys_pre_rope=True)
    if r.integers(4) == 0:
        w = synth.compress_pool(w)
    opts = dict(rows_per_block=int(r.choice([0, 0, 64, 128, 256])),
                kv_splits=int(r.choice([0, 0, 1, 3])), page_size=int(r.choice([64, 128])))
    return w, opts


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_configuration(i):
    w, opts = _case(i)
    what = (f"random {i}: {w.pool_dtype} H {w.n_q_heads}/{w.n_kv_heads} d {w.head_dim} "
            f"B {w.batch} S {w.suffix_len} pre_rope {w.keys_pre_rope} "
            f"compressed {w.pool_compressed} {opts}")
    say(what)
    ref_out, ref_lse, _ = oracle_ref(w)
    out, lse, plan, dev = run_fused(w, **opts)
    compare(w, out, lse, ref_out, ref_lse, what=f"{what}/fused")
    out2, lse2, _, _, _ = run_paged(w, dev=dev, plan=plan)
    compare(w, out2, lse2, ref_out, ref_lse, what=f"{what}/paged")
    assert torch.equal(out, out2), what
