"""Extraction-time attention with Structured Information Flow (Section 3.3)
through the C ABI (c2kv_sif_plan_create + c2kv_attend) against the float64
oracle, over several shapes, edge cases and launch shapes."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_17715_amd as c2kv
import synth
from gpu_common import compare, say

pytestmark = pytest.mark.gpu


def _run(w, **opts):
    plan = c2kv.Plan.for_sif(w, **opts).upload()
    q = c2kv.to_device(w.q, w.act_dtype)
    k = c2kv.to_device(w.k, w.act_dtype)
    v = c2kv.to_device(w.v, w.act_dtype)
    out = torch.empty_like(q)
    lse = torch.empty((w.batch, w.n_q_heads, w.seq_len), dtype=torch.float32, device="cuda")
    c2kv.c2kv_attend(plan, None, None, q, k, v, out, lse)
    torch.cuda.synchronize()
    return out, lse, plan


def _ref(w):
    outs, lses = [], []
    for b in range(w.batch):
        q, k, v = (oracle.decode_storage(x[b], w.act_dtype) for x in (w.q, w.k, w.v))
        o, l = oracle.sif_attend(q, k, v, w.n_tokens, w.block, w.sink, w.rope_base)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses)


CASES = [
    dict(act_dtype="bf16", n_tokens=300, block=4, sink=4, n_q_heads=8, n_kv_heads=2),
    dict(act_dtype="f32", n_tokens=130, block=3, sink=0, n_q_heads=4, n_kv_heads=2,
         head_dim=64),
    dict(act_dtype="bf16", n_tokens=512, block=4, sink=4, n_q_heads=32, n_kv_heads=8),
    dict(act_dtype="bf16", n_tokens=50, block=64, sink=2, n_q_heads=8, n_kv_heads=2),
    dict(act_dtype="bf16", n_tokens=70, block=1, sink=1, n_q_heads=8, n_kv_heads=2),
    dict(act_dtype="bf16", n_tokens=40, block=8, sink=40, n_q_heads=8, n_kv_heads=2),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_sif_matches_oracle(case):
    w = synth.sif(batch=2, seed=900 + case, **CASES[case])
    say(f"sif case {case}: {CASES[case]}")
    out, lse, plan = _run(w)
    ref_out, ref_lse = _ref(w)
    compare(w, out, lse, ref_out, ref_lse, what=f"sif-{case}")


@pytest.mark.parametrize("opts", [dict(rows_per_block=128), dict(rows_per_block=64),
                                  dict(rows_per_block=256), dict(kv_splits=2),
                                  dict(rows_per_block=128, kv_splits=3)])
def test_sif_launch_shapes_agree(opts):
    w = synth.sif(batch=2, n_tokens=300, block=4, sink=4, n_q_heads=8, n_kv_heads=2, seed=950)
    ref_out, ref_lse = _ref(w)
    out, lse, _ = _run(w, **opts)
    compare(w, out, lse, ref_out, ref_lse, what=f"sif {opts}")


def test_sif_original_rows_are_plain_causal_attention():
    """Original-token invariance on the GPU: changing the C^2 tokens' keys and
    values leaves every original row's output bit-identical."""
    w = synth.sif(batch=1, n_tokens=256, block=4, sink=4, n_q_heads=8, n_kv_heads=2, seed=960)
    out, _, _ = _run(w)
    n = w.n_tokens
    k2, v2 = w.k.copy(), w.v.copy()
    k2[:, n:] = w.k[:, n:][:, ::-1]
    v2[:, n:] = w.v[:, n:][:, ::-1]
    out2, _, _ = _run(synth.dataclasses.replace(w, k=k2, v=v2))
    assert torch.equal(out[:, :n], out2[:, :n])
    assert not torch.equal(out[:, n:], out2[:, n:])


@pytest.mark.parametrize("i", range(24))
def test_sif_random_configurations(i):
    """Seeded random SIF shapes: sequence length, block size (including blocks
    longer than the sequence), sink, heads, head size, dtype and launch shape."""
    r = np.random.default_rng(9100 + i)
    n = int(r.integers(1, 400))
    kw = dict(n_tokens=n, block=int(r.choice([1, 2, 3, 4, 8, 64, 500])),
              sink=int(r.integers(0, min(n, 70) + 1)),
              act_dtype=["bf16", "bf16", "f32"][r.integers(3)],
              head_dim=int(r.choice([64, 128])))
    hq, hkv = [(8, 2), (4, 4), (16, 4), (8, 1)][r.integers(4)]
    opts = dict(rows_per_block=int(r.choice([0, 64, 128, 256])), kv_splits=int(r.choice([0, 0, 2])))
    w = synth.sif(batch=int(r.integers(1, 3)), n_q_heads=hq, n_kv_heads=hkv, seed=9200 + i, **kw)
    say(f"sif random {i}: {kw} H {hq}/{hkv} {opts}")
    ref_out, ref_lse = _ref(w)
    out, lse, _ = _run(w, **opts)
    compare(w, out, lse, ref_out, ref_lse, what=f"sif random {i}")
