"""Pins of the float64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: a worked
example of the placement rule, closed forms, the complex-number form of RoPE,
textbook causal attention through torch's SDPA, scalar brute force, exact
rationals, and invariances.  A dropped term, a wrong sign or index, a swapped
operand or an off-by-one in the causal mask fails at least one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# layout: span-preserving placement (Section 3.2, "Output and Reuse")
# ---------------------------------------------------------------------------

def test_layout_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "layout_worked_example.json")))
    lay = oracle.compose_layout(g["req_seg_off"], g["seg_row0"], g["seg_span"],
                                g["seg_orig_pos0"], g["seg_kept_off"], g["kept_idx"])
    for key in ("src_row", "p_new", "p_orig", "delta", "seg"):
        got = [list(map(int, a)) for a in lay[key]]
        assert got == g["expect"][key], key
    assert list(map(int, lay["span_end"])) == g["expect"]["span_end"]
    assert list(map(int, lay["composed_len"])) == g["expect"]["composed_len"]


def test_layout_explicit_placement_worked_example():
    """Explicit placements out of order and overlapping, one segment keeping
    nothing, negative deltas: the hand-worked values, including span_end as the
    first position past every placed span (not the last segment's span end)."""
    g = json.load(open(os.path.join(GOLDEN, "layout_explicit_placement.json")))
    lay = oracle.compose_layout(g["req_seg_off"], g["seg_row0"], g["seg_span"],
                                g["seg_orig_pos0"], g["seg_kept_off"], g["kept_idx"],
                                seg_new_pos0=g["seg_new_pos0"])
    for key in ("src_row", "p_new", "p_orig", "delta", "seg"):
        got = [list(map(int, a)) for a in lay[key]]
        assert got == g["expect"][key], key
    assert list(map(int, lay["span_end"])) == g["expect"]["span_end"]
    assert list(map(int, lay["composed_len"])) == g["expect"]["composed_len"]
    # the case the pin exists for: the last segment is not the furthest
    assert g["expect"]["span_end"] != g["expect"]["last_segment_span_end"]


def test_span_end_is_past_every_covered_position():
    """Independent construction of span_end for explicit placements: mark every
    position that any segment's uncompressed span covers, token by token; the
    first query position is one past the largest marked position, and no cached
    slot sits at or after it."""
    rng = np.random.default_rng(77)
    for _ in range(200):
        nseg = int(rng.integers(1, 6))
        span = rng.integers(1, 9, nseg)
        new0 = rng.integers(0, 40, nseg)
        kept = [np.sort(rng.choice(int(s), size=int(rng.integers(0, s + 1)), replace=False))
                for s in span]
        koff = np.concatenate([[0], np.cumsum([len(k) for k in kept])])
        lay = oracle.compose_layout([0, nseg], np.zeros(nseg, int), span,
                                    np.zeros(nseg, int), koff,
                                    np.concatenate(kept + [np.zeros(0, int)]),
                                    seg_new_pos0=new0)
        covered = set()
        for c in range(nseg):
            covered.update(range(int(new0[c]), int(new0[c] + span[c])))
        expect = max(covered) + 1
        assert int(lay["span_end"][0]) == expect
        assert all(int(p) < expect for p in lay["p_new"][0])


def _layout_by_loops(w):
    """Second, independent enumeration: positions from a running cursor over
    every uncompressed token of every segment (kept or not)."""
    res = []
    for r in range(len(w.req_seg_off) - 1):
        cursor = 0
        slots = []
        for c in range(w.req_seg_off[r], w.req_seg_off[r + 1]):
            kept = set(int(x) for x in w.kept_idx[w.seg_kept_off[c]:w.seg_kept_off[c + 1]])
            for j in range(int(w.seg_span[c])):      # walk the whole span
                if j in kept:
                    slots.append((int(w.seg_row0[c]) + j, cursor,
                                  cursor - (int(w.seg_orig_pos0[c]) + j)))
                cursor += 1
        res.append((slots, cursor))
    return res


@pytest.mark.parametrize("idx", [1, 2])
def test_layout_matches_token_walk(idx):
    w = synth.config(idx)
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx)
    for r, (slots, end) in enumerate(_layout_by_loops(w)):
        assert [s[0] for s in slots] == list(map(int, lay["src_row"][r]))
        assert [s[1] for s in slots] == list(map(int, lay["p_new"][r]))
        assert [s[2] for s in slots] == list(map(int, lay["delta"][r]))
        assert end == int(lay["span_end"][r])


def test_layout_ragged_matches_token_walk():
    w = synth.small(keep=("ratio", 0.0, 0.3), batch=3, chunks_per_req=4)
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx)
    for r, (slots, end) in enumerate(_layout_by_loops(w)):
        assert [s[1] for s in slots] == list(map(int, lay["p_new"][r]))
        assert end == int(lay["span_end"][r])


def test_c2_token_positions():
    """Section 3.2.1: m = ceil(n/k) memory slots; Section 3.3.1: block
    B(j) = {(j-1)k+1, ..., min(jk, n)} (1-based) and slot j takes the position
    of the last token of its block -> 0-based index min(jk, n) - 1."""
    for n, k, want in [(10, 4, [3, 7, 9]), (8, 4, [3, 7]), (5, 8, [4]), (1, 4, [0]),
                       (512, 4, list(range(3, 512, 4)))]:
        got = synth._kept_for_chunk(None, ("c2", k), n)
        assert list(map(int, got)) == want
        assert len(got) == -(-n // k)


# ---------------------------------------------------------------------------
# RoPE
# ---------------------------------------------------------------------------

def _rope_complex(x, pos, base):
    """Independent form: pair (x_i, x_{i+d/2}) as the complex number
    x_i + i x_{i+d/2}, multiplied by exp(i * pos * base^(-2i/d))."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    z = x[..., :h] + 1j * x[..., h:]
    freq = np.array([base ** (-(2.0 * i) / d) for i in range(h)])
    z = z * np.exp(1j * np.asarray(pos, np.float64)[..., None] * freq)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rope_matches_complex_form():
    rng = np.random.default_rng(0)
    for d, base in [(64, 1e4), (128, 5e5), (4, 10.0)]:
        x = rng.standard_normal((50, d))
        pos = rng.integers(-70000, 70000, size=50)
        np.testing.assert_allclose(oracle.rope_rotate(x, pos, base),
                                   _rope_complex(x, pos, base), atol=1e-9, rtol=0)


def test_rope_d2_closed_form():
    """d = 2: theta_0 = 1, so position p is the plane rotation by p radians."""
    for p in [1, 2, -3, 1000]:
        R = np.array([[math.cos(p), -math.sin(p)], [math.sin(p), math.cos(p)]])
        for x in ([1.0, 0.0], [0.0, 1.0], [0.3, -2.0]):
            np.testing.assert_allclose(oracle.rope_rotate(np.array(x), p, 7.0),
                                       R @ np.array(x), atol=1e-12)


def test_rope_d4_frequencies():
    """d = 4, base 100: theta = (1, 1/10); pairs (x0, x2) and (x1, x3)."""
    x = np.array([1.0, 2.0, 3.0, 4.0])
    p = 5
    a, b = p * 1.0, p * 0.1
    want = [1 * math.cos(a) - 3 * math.sin(a), 2 * math.cos(b) - 4 * math.sin(b),
            1 * math.sin(a) + 3 * math.cos(a), 2 * math.sin(b) + 4 * math.cos(b)]
    np.testing.assert_allclose(oracle.rope_rotate(x, p, 100.0), want, atol=1e-12)


def test_rope_group_laws():
    """Invariant 1: R(delta) R(p) = R(p + delta); R(0) = I; R(-p) R(p) = I;
    each pair keeps its norm; scores depend only on relative position."""
    rng = np.random.default_rng(1)
    d, base = 128, 5e5
    x = rng.standard_normal((64, d))
    p = rng.integers(0, 70000, 64)
    dl = rng.integers(-70000, 70000, 64)
    np.testing.assert_allclose(oracle.rope_rotate(oracle.rope_rotate(x, p, base), dl, base),
                               oracle.rope_rotate(x, p + dl, base), atol=1e-9)
    np.testing.assert_array_equal(oracle.rope_rotate(x, np.zeros(64), base), x)
    np.testing.assert_allclose(oracle.rope_rotate(oracle.rope_rotate(x, p, base), -p, base),
                               x, atol=1e-9)
    y = oracle.rope_rotate(x, p, base)
    np.testing.assert_allclose(x[:, :64] ** 2 + x[:, 64:] ** 2,
                               y[:, :64] ** 2 + y[:, 64:] ** 2, atol=1e-9)
    q = rng.standard_normal((64, d))
    a = rng.integers(0, 70000, 64)
    b = rng.integers(0, 70000, 64)
    lhs = np.sum(oracle.rope_rotate(q, a, base) * oracle.rope_rotate(x, b, base), -1)
    rhs = np.sum(q * oracle.rope_rotate(x, b - a, base), -1)
    np.testing.assert_allclose(lhs, rhs, atol=1e-8)


# ---------------------------------------------------------------------------
# attention: composition equals concatenation (Section 3.2; Eq. 3-4)
# ---------------------------------------------------------------------------

def _sdpa_reference(keys_pos, vals, q_pre, q_pos, n_cached, Hq, Hkv):
    """torch SDPA in float64 over the full key sequence with an explicit
    bottom-right causal mask and the library's own GQA head mapping."""
    S = q_pre.shape[0]
    L = keys_pos.shape[0]
    qt = torch.from_numpy(q_pre).permute(1, 0, 2)[None]        # [1, Hq, S, d]
    kt = torch.from_numpy(keys_pos).permute(1, 0, 2)[None]     # [1, Hkv, L, d]
    vt = torch.from_numpy(vals).permute(1, 0, 2)[None]
    mask = torch.ones(S, L, dtype=torch.bool)
    for t in range(S):
        mask[t, n_cached + t + 1:] = False
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask,
                                                         enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()                       # [S, Hq, d]


def _keep_all_workload(seed):
    """All tokens kept, float32 storage; chunk keys encoded either at their final
    positions (delta 0) or at 0.. (delta = placement)."""
    w = synth.small(pool_dtype="f32", keep=("all",), n_pool_chunks=3, chunk_len=11,
                    prefix_len=5, batch=1, chunks_per_req=3, suffix_len=6, head_dim=16,
                    n_q_heads=6, n_kv_heads=2, seed=seed, order="shuffled")
    return w


@pytest.mark.parametrize("seed", [3, 4])
def test_keep_all_delta0_equals_full_causal_attention(seed):
    """Invariant 2: keep-ratio 1, no quantisation, segments already encoded at
    their final positions -> plain causal attention over the concatenation."""
    w = _keep_all_workload(seed)
    base = w.rope_base
    lay = oracle.compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                                w.seg_kept_off, w.kept_idx)
    # re-encode: make each stored key sit at its final position (orig_pos0 = new_pos0)
    new0 = []
    pos = 0
    for c in range(w.n_segments):
        new0.append(pos)
        pos += int(w.seg_span[c])
    w2 = synth.with_overrides(w, seg_orig_pos0=np.array(new0, np.int32))
    out, lse, lay2 = oracle.compose_attend(w2)
    assert all(int(d) == 0 for d in lay2["delta"][0])

    # reference: the raw sequence [prefix, chunks in order, suffix]
    rows = lay["src_row"][0]
    kc = w.pool_k[rows].astype(np.float64)
    vc = w.pool_v[rows].astype(np.float64)
    N = len(rows)
    S = w.suffix_len
    se = int(lay["span_end"][0])
    ks = _rope_complex(w.k_suf[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    keys = np.concatenate([kc, ks], 0)
    vals = np.concatenate([vc, w.v_suf[0].astype(np.float64)], 0)
    qp = _rope_complex(w.q[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    ref = _sdpa_reference(keys, vals, qp, None, N, w.n_q_heads, w.n_kv_heads)
    np.testing.assert_allclose(out[0], ref, atol=1e-12, rtol=0)


@pytest.mark.parametrize("seed", [5, 6])
def test_rerotation_equals_encoding_at_global_positions(seed):
    """Invariants 1 + 2: chunks stored at positions 0.. and re-rotated give the
    same attention as un-rotated keys encoded directly at their global positions."""
    w = _keep_all_workload(seed)
    base = w.rope_base
    out, _, lay = oracle.compose_attend(w)
    rows = lay["src_row"][0]
    # the pool holds keys encoded at p_orig; recover the un-rotated key, then
    # encode it at the global position with the complex form
    k_enc = w.pool_k[rows].astype(np.float64)
    k_raw = _rope_complex(k_enc, -lay["p_orig"][0][:, None].astype(np.float64), base)
    k_glob = _rope_complex(k_raw, lay["p_new"][0][:, None].astype(np.float64), base)
    vc = w.pool_v[rows].astype(np.float64)
    S = w.suffix_len
    se = int(lay["span_end"][0])
    ks = _rope_complex(w.k_suf[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    qp = _rope_complex(w.q[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    ref = _sdpa_reference(np.concatenate([k_glob, ks]), np.concatenate([vc, w.v_suf[0]]),
                          qp, None, len(rows), w.n_q_heads, w.n_kv_heads)
    np.testing.assert_allclose(out[0], ref, atol=1e-10, rtol=0)


@pytest.mark.parametrize("seed,keep", [(7, ("all",)), (8, ("ratio", 0.2, 0.7)),
                                       (9, ("c2", 4))])
def test_pre_rope_keys_encoded_at_new_positions(seed, keep):
    """Keys stored before positional encoding (Section 3.3.1): each kept key is
    encoded at its new position, checked against the complex form of RoPE and
    torch's SDPA over [composed keys | suffix]."""
    w = synth.small(pool_dtype="f32", keep=keep, n_pool_chunks=3, chunk_len=11,
                    prefix_len=5, batch=1, chunks_per_req=3, suffix_len=6, head_dim=16,
                    n_q_heads=6, n_kv_heads=2, seed=seed, order="shuffled")
    w = synth.with_overrides(w, keys_pre_rope=True)
    base = w.rope_base
    out, _, lay = oracle.compose_attend(w)
    rows = lay["src_row"][0]
    k_glob = _rope_complex(w.pool_k[rows].astype(np.float64),
                           lay["p_new"][0][:, None].astype(np.float64), base)
    vc = w.pool_v[rows].astype(np.float64)
    S = w.suffix_len
    se = int(lay["span_end"][0])
    ks = _rope_complex(w.k_suf[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    qp = _rope_complex(w.q[0].astype(np.float64), (se + np.arange(S))[:, None], base)
    ref = _sdpa_reference(np.concatenate([k_glob, ks]), np.concatenate([vc, w.v_suf[0]]),
                          qp, None, len(rows), w.n_q_heads, w.n_kv_heads)
    np.testing.assert_allclose(out[0], ref, atol=1e-10, rtol=0)
    # and it is not the delta reading of the same stored values
    other, _, _ = oracle.compose_attend(synth.with_overrides(w, keys_pre_rope=False))
    assert np.abs(other - out).max() > 1e-3


@pytest.mark.parametrize("keep", [("ratio", 0.1, 0.6), ("c2", 4), ("none",)])
def test_compressed_pool_reads_the_same_tokens(keep):
    """A chunk stored compressed (Section 3.2: only its kept tokens are saved)
    holds the k-th kept token in row k: the composed result equals that of the
    whole chunk with kept index j in row j, for every request of a batch that
    reuses chunks."""
    w = synth.small(pool_dtype="f32", keep=keep, batch=3, n_pool_chunks=4, chunks_per_req=3,
                    head_dim=16, n_q_heads=4, n_kv_heads=2, suffix_len=5, chunk_len=40)
    wc = synth.compress_pool(w)
    assert wc.pool_k.shape[0] == sum(
        len(set(map(int, w.kept_idx[w.seg_kept_off[c]:w.seg_kept_off[c + 1]])))
        for c in sorted({int(r): i for i, r in enumerate(w.seg_row0)}.values()))
    a, la, _ = oracle.compose_attend(w)
    b, lb, _ = oracle.compose_attend(wc)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)


def test_fixed_pos_ablation_differs():
    """Section 4.8 (Fixed-Pos): without re-rotation the result changes."""
    w = synth.small(pool_dtype="f32", head_dim=16, suffix_len=4, batch=1)
    a, _, _ = oracle.compose_attend(w)
    b, _, _ = oracle.compose_attend(w, rerotate=False)
    assert np.abs(a - b).max() > 1e-3


# ---------------------------------------------------------------------------
# softmax rows, LSE
# ---------------------------------------------------------------------------

def test_rows_sum_to_one_and_lse():
    """Invariant 3 and the log-sum-exp of the scaled scores (scipy)."""
    from scipy.special import logsumexp
    rng = np.random.default_rng(7)
    N, S, Hq, Hkv, d = 9, 5, 4, 2, 8
    kc, vc = rng.standard_normal((N, Hkv, d)), rng.standard_normal((N, Hkv, d))
    q, ks, vs = (rng.standard_normal((S, Hq, d)), rng.standard_normal((S, Hkv, d)),
                 rng.standard_normal((S, Hkv, d)))
    out, lse, p = oracle.attend(kc, vc, q, ks, vs, 20, 1e4, return_probs=True)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-12)
    # causal: suffix key u is invisible to suffix row t < u
    for t in range(S):
        assert np.all(p[:, t, N + t + 1:] == 0)
        assert np.all(p[:, t, :N + t + 1] > 0)
    # lse vs scipy on independently formed scores
    qr = _rope_complex(q, (20 + np.arange(S))[:, None], 1e4)
    kr = _rope_complex(ks, (20 + np.arange(S))[:, None], 1e4)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        for t in range(S):
            sc = [float(qr[t, h] @ kc[j, g]) / math.sqrt(d) for j in range(N)]
            sc += [float(qr[t, h] @ kr[u, g]) / math.sqrt(d) for u in range(t + 1)]
            assert abs(lse[h, t] - logsumexp(sc)) < 1e-12


# ---------------------------------------------------------------------------
# brute force on 2-token chunks (Invariant 4)
# ---------------------------------------------------------------------------

def _brute(chunks, order, kept_sets, q, ks, vs, base):
    """Scalar loops: assemble every visible key with its absolute position, rotate
    with explicit cos/sin per pair, softmax with math.exp."""
    d = len(q[0][0])
    h2 = d // 2
    theta = [base ** (-2.0 * i / d) for i in range(h2)]

    def rot(x, p):
        y = [0.0] * d
        for i in range(h2):
            c, s = math.cos(p * theta[i]), math.sin(p * theta[i])
            y[i] = x[i] * c - x[i + h2] * s
            y[i + h2] = x[i] * s + x[i + h2] * c
        return y

    keys, vals = [], []
    cursor = 0
    for ci in order:
        kk, vv = chunks[ci]
        for j in range(2):
            if j in kept_sets[ci]:
                # stored key was encoded at position j; it must end at cursor + j
                # stored key was encoded at position j: undo that, encode at cursor + j
                keys.append(rot(rot(kk[j], -j), cursor + j))
                vals.append(vv[j])
        cursor += 2
    S = len(q)
    Hq = len(q[0])
    out = [[None] * Hq for _ in range(S)]
    for t in range(S):
        for h in range(Hq):
            g = 0
            qt = rot(q[t][h], cursor + t)
            kl = keys + [rot(ks[u][g], cursor + u) for u in range(t + 1)]
            vl = vals + [vs[u][g] for u in range(t + 1)]
            sc = [sum(a * b for a, b in zip(qt, k)) / math.sqrt(d) for k in kl]
            m = max(sc)
            e = [math.exp(x - m) for x in sc]
            z = sum(e)
            out[t][h] = [sum(e[j] * vl[j][i] for j in range(len(vl))) / z for i in range(d)]
    return out


def test_brute_force_two_token_chunks():
    rng = np.random.default_rng(11)
    d, Hq, base = 4, 2, 10.0
    # float32-representable values: the pool below is declared as fp32 storage
    chunks = [(rng.standard_normal((2, d)).astype(np.float32).astype(np.float64),
               rng.standard_normal((2, d)).astype(np.float32).astype(np.float64))
              for _ in range(3)]
    subsets = [set(), {0}, {1}, {0, 1}]
    n_cases = 0
    for n_ch in (1, 2, 3):
        for order in itertools.permutations(range(3), n_ch):
            for ks_choice in itertools.product(range(4), repeat=n_ch):
                if n_cases % 7 and n_ch == 3:      # thin the 3-chunk orders
                    n_cases += 1
                    continue
                n_cases += 1
                kept_sets = {order[i]: subsets[ks_choice[i]] for i in range(n_ch)}
                S = 1 + (n_cases % 2)
                q = rng.standard_normal((S, Hq, d))
                ksf = rng.standard_normal((S, 1, d))
                vsf = rng.standard_normal((S, 1, d))
                # pool: chunk c at rows 2c, 2c+1, each encoded at positions 0, 1
                pool_k = np.stack([chunks[c][0] for c in range(3)]).reshape(6, 1, d)
                pool_v = np.stack([chunks[c][1] for c in range(3)]).reshape(6, 1, d)
                kept = []
                off = [0]
                for c in order:
                    kept += sorted(kept_sets[c])
                    off.append(len(kept))
                lay = oracle.compose_layout([0, n_ch], [2 * c for c in order], [2] * n_ch,
                                            [0] * n_ch, off, kept)
                (kc, vc), = oracle.compose(lay, pool_k, pool_v, "f32", base)
                out, _ = oracle.attend(kc, vc, q, ksf, vsf, int(lay["span_end"][0]), base)
                want = _brute([(c[0].tolist(), c[1].tolist()) for c in chunks], order,
                              {c: kept_sets[c] for c in order}, q.tolist(),
                              ksf[:, 0:1, :].tolist(), vsf.tolist(), base)
                np.testing.assert_allclose(out, np.array(want), atol=1e-12)
    assert n_cases > 100


def test_closed_forms():
    """One cached key and S = 1: two keys, p0 = sigmoid(s0 - s1).
    All keys equal: output = mean of the values."""
    rng = np.random.default_rng(12)
    d = 8
    kc, vc = rng.standard_normal((1, 1, d)), rng.standard_normal((1, 1, d))
    q, ks, vs = (rng.standard_normal((1, 1, d)), rng.standard_normal((1, 1, d)),
                 rng.standard_normal((1, 1, d)))
    base, se = 1e4, 3
    out, lse, p = oracle.attend(kc, vc, q, ks, vs, se, base, return_probs=True)
    qr = _rope_complex(q[0, 0], se, base)
    s0 = qr @ kc[0, 0] / math.sqrt(d)
    s1 = qr @ _rope_complex(ks[0, 0], se, base) / math.sqrt(d)
    p0 = 1.0 / (1.0 + math.exp(-(s0 - s1)))
    assert abs(p[0, 0, 0] - p0) < 1e-14
    np.testing.assert_allclose(out[0, 0], p0 * vc[0, 0] + (1 - p0) * vs[0, 0], atol=1e-14)
    # every score equal (zero query): the output is the mean of all visible values
    N = 7
    kc = np.tile(rng.standard_normal((1, 1, d)), (N, 1, 1))
    vc = rng.standard_normal((N, 1, d))
    q = np.zeros((1, 1, d))        # zero query: every score is 0
    out, _ = oracle.attend(kc, vc, q, ks, vs, 10, base)
    np.testing.assert_allclose(out[0, 0], (vc[:, 0].sum(0) + vs[0, 0]) / (N + 1), atol=1e-14)


# ---------------------------------------------------------------------------
# set semantics of the composed cache; split / merge
# ---------------------------------------------------------------------------

def test_cached_slot_permutation_invariance():
    rng = np.random.default_rng(13)
    N, S, Hq, Hkv, d = 40, 6, 4, 2, 16
    kc, vc = rng.standard_normal((N, Hkv, d)), rng.standard_normal((N, Hkv, d))
    q, ks, vs = (rng.standard_normal((S, Hq, d)), rng.standard_normal((S, Hkv, d)),
                 rng.standard_normal((S, Hkv, d)))
    a, la = oracle.attend(kc, vc, q, ks, vs, 100, 1e4)
    perm = rng.permutation(N)
    b, lb = oracle.attend(kc[perm], vc[perm], q, ks, vs, 100, 1e4)
    np.testing.assert_allclose(a, b, atol=1e-12)
    np.testing.assert_allclose(la, lb, atol=1e-12)


def test_split_merge_equals_whole():
    """Attention over a partition of the cached keys, merged by log-sum-exp,
    equals attention over all keys (the split-K combine)."""
    rng = np.random.default_rng(14)
    N, S, Hq, Hkv, d = 50, 4, 4, 1, 8
    kc, vc = rng.standard_normal((N, Hkv, d)), rng.standard_normal((N, Hkv, d))
    q, ks, vs = (rng.standard_normal((S, Hq, d)), rng.standard_normal((S, Hkv, d)),
                 rng.standard_normal((S, Hkv, d)))
    whole, lw = oracle.attend(kc, vc, q, ks, vs, 60, 1e4)
    # parts: cached slots in 3 groups (the suffix goes with the last group);
    # for the first groups, hide the suffix by giving those calls no visible suffix:
    # build them with scores directly
    cuts = [0, 17, 31, N]
    parts = []
    qr = _rope_complex(q, (60 + np.arange(S))[:, None], 1e4)
    kr = _rope_complex(ks, (60 + np.arange(S))[:, None], 1e4)
    for i in range(3):
        lo, hi = cuts[i], cuts[i + 1]
        o = np.zeros((S, Hq, d)); l = np.zeros((S, Hq))
        for h in range(Hq):
            keys = kc[lo:hi, 0]; vals = vc[lo:hi, 0]
            sc = qr[:, h] @ keys.T / math.sqrt(d)
            if i == 2:
                ssuf = qr[:, h] @ kr[:, 0].T / math.sqrt(d)
                ssuf = np.where(np.tril(np.ones((S, S))) > 0, ssuf, -np.inf)
                sc = np.concatenate([sc, ssuf], 1)
                vals = np.concatenate([vals, vs[:, 0]], 0)
            m = sc.max(1, keepdims=True)
            e = np.exp(sc - m)
            o[:, h] = e @ vals / e.sum(1, keepdims=True)
            l[:, h] = m[:, 0] + np.log(e.sum(1))
        parts.append((o, l))
    mo, ml = oracle.merge_partials(parts)
    np.testing.assert_allclose(mo, whole, atol=1e-12)
    np.testing.assert_allclose(ml.T, lw, atol=1e-12)


def test_gqa_head_mapping():
    """Query head h reads kv-head h // G: consecutive query heads share a kv-head."""
    rng = np.random.default_rng(15)
    N, S, Hq, Hkv, d = 5, 2, 6, 3, 4
    kc, vc = rng.standard_normal((N, Hkv, d)), rng.standard_normal((N, Hkv, d))
    q, ks, vs = (rng.standard_normal((S, Hq, d)), rng.standard_normal((S, Hkv, d)),
                 rng.standard_normal((S, Hkv, d)))
    out, _ = oracle.attend(kc, vc, q, ks, vs, 9, 1e4)
    for h in range(Hq):
        g = h // 2
        o1, _ = oracle.attend(kc[:, g:g + 1], vc[:, g:g + 1], q[:, h:h + 1],
                              ks[:, g:g + 1], vs[:, g:g + 1], 9, 1e4)
        np.testing.assert_allclose(out[:, h], o1[:, 0], atol=1e-14)


# ---------------------------------------------------------------------------
# storage decode
# ---------------------------------------------------------------------------

def test_int8_decode_exact():
    rng = np.random.default_rng(16)
    codes = rng.integers(-127, 128, size=(20, 3, 8)).astype(np.int8)
    scale = (rng.random((20, 3)) * 0.05).astype(np.float32)
    x = oracle.decode_storage(codes, "i8", scale)
    for (i, j, k), v in np.ndenumerate(x):
        assert Fraction(v) == Fraction(int(codes[i, j, k])) * Fraction(float(scale[i, j]))


def test_bf16_decode_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0001, 0x7F7F, 0x0000, 0x8000], np.uint16)
    want = [1.0, -1.0, 3.140625, 2.0 ** -133, 3.3895313892515355e38, 0.0, -0.0]
    got = oracle.decode_bf16(bits)
    for g, w_ in zip(got, want):
        assert g == w_
    # round trip with the generator's RNE cast
    rng = np.random.default_rng(17)
    x = rng.standard_normal(1000).astype(np.float32)
    b = synth.f32_to_bf16_bits(x)
    assert np.all(np.abs(oracle.decode_bf16(b) - x) <= np.abs(x) * 2.0 ** -8)


def test_generator_bf16_paths_agree():
    rng = np.random.default_rng(18)
    x = (rng.standard_normal(1 << 17) * 5).astype(np.float32)
    np.testing.assert_array_equal(synth.f32_to_bf16_bits(x), synth.f32_to_bf16_bits_int(x))


# ---------------------------------------------------------------------------
# extraction-time attention with Structured Information Flow (Section 3.3)
# ---------------------------------------------------------------------------

def test_sif_worked_example():
    """n = 5 originals, blocks of 2, a 1-token sink: blocks {0,1}, {2,3}, {4};
    C^2 tokens at the positions of their blocks' last tokens 1, 3, 4."""
    np.testing.assert_array_equal(oracle.sif_positions(5, 2), [0, 1, 2, 3, 4, 1, 3, 4])
    #               o0 o1 o2 o3 o4 c0 c1 c2
    want = np.array([[1, 0, 0, 0, 0, 0, 0, 0],
                     [1, 1, 0, 0, 0, 0, 0, 0],
                     [1, 1, 1, 0, 0, 0, 0, 0],
                     [1, 1, 1, 1, 0, 0, 0, 0],
                     [1, 1, 1, 1, 1, 0, 0, 0],
                     [1, 1, 0, 0, 0, 1, 0, 0],      # c0: its block {0, 1}, sink {0}
                     [1, 0, 1, 1, 0, 1, 1, 0],      # c1: {2, 3}, sink, c0..c1
                     [1, 0, 0, 0, 1, 1, 1, 1]], bool)
    np.testing.assert_array_equal(oracle.sif_mask(5, 2, 1), want)


def _sif_reference(q, k, v, n, block, sink, base):
    """Independent construction: visible key sets per row from the definitions
    (1-based blocks B(j) = {(j-1)k+1, ..., min(jk, n)}), C^2 positions from each
    block's last member, complex-form RoPE, torch SDPA with the boolean mask."""
    m = -(-n // block)
    blocks = [list(range((j - 1) * block + 1, min(j * block, n) + 1)) for j in range(1, m + 1)]
    pos = list(range(n)) + [max(b) - 1 for b in blocks]         # 0-based positions
    L = n + m
    mask = torch.zeros(L, L, dtype=torch.bool)
    for t in range(1, n + 1):                                     # original x_t (1-based)
        for u in range(1, t + 1):
            mask[t - 1, u - 1] = True
    for j in range(1, m + 1):                                     # C^2 token c_j
        row = n + j - 1
        for u in set(blocks[j - 1]) | set(range(1, sink + 1)):
            mask[row, u - 1] = True
        for jj in range(1, j + 1):
            mask[row, n + jj - 1] = True
    P = np.array(pos, np.float64)[:, None]
    qp = _rope_complex(q, P, base)
    kp = _rope_complex(k, P, base)
    qt = torch.from_numpy(qp).permute(1, 0, 2)[None]
    kt = torch.from_numpy(kp).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.asarray(v, np.float64)).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask,
                                                         enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("n,block,sink", [(13, 4, 0), (13, 4, 2), (8, 8, 3), (9, 1, 1),
                                          (7, 10, 7)])
def test_sif_matches_independent_construction(n, block, sink):
    w = synth.sif(batch=1, n_tokens=n, block=block, sink=sink, n_q_heads=4, n_kv_heads=2,
                  head_dim=8, act_dtype="f32", seed=n * 100 + block * 10 + sink)
    q, k, v = (x[0].astype(np.float64) for x in (w.q, w.k, w.v))
    out, lse = oracle.sif_attend(q, k, v, n, block, sink, w.rope_base)
    ref = _sif_reference(q, k, v, n, block, sink, w.rope_base)
    np.testing.assert_allclose(out, ref, atol=1e-10, rtol=0)
    assert np.isfinite(lse).all()


def test_sif_original_token_invariance_and_locality():
    """Original rows are plain causal attention over the originals and ignore
    every C^2 token; a C^2 row ignores originals outside its block and the sink
    and later C^2 tokens, and does see its own block."""
    n, block, sink = 20, 4, 2
    w = synth.sif(batch=1, n_tokens=n, block=block, sink=sink, n_q_heads=4, n_kv_heads=2,
                  head_dim=8, act_dtype="f32", seed=77)
    q, k, v = (x[0].astype(np.float64).copy() for x in (w.q, w.k, w.v))
    out, _ = oracle.sif_attend(q, k, v, n, block, sink, w.rope_base)
    # originals: torch causal SDPA over the first n tokens only
    P = np.arange(n, dtype=np.float64)[:, None]
    qt = torch.from_numpy(_rope_complex(q[:n], P, w.rope_base)).permute(1, 0, 2)[None]
    kt = torch.from_numpy(_rope_complex(k[:n], P, w.rope_base)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v[:n]).permute(1, 0, 2)[None]
    causal = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True,
                                                              enable_gqa=True)
    np.testing.assert_allclose(out[:n], causal[0].permute(1, 0, 2).numpy(), atol=1e-10, rtol=0)
    rng = np.random.default_rng(5)
    # perturbing C^2 tokens leaves the original rows as they are
    k2, v2 = k.copy(), v.copy()
    k2[n:] += rng.standard_normal(k2[n:].shape)
    v2[n:] += rng.standard_normal(v2[n:].shape)
    o2, _ = oracle.sif_attend(q, k2, v2, n, block, sink, w.rope_base)
    np.testing.assert_array_equal(o2[:n], out[:n])
    # C^2 token j = 2 (block {8..11}): originals 4..7 and 12.. and C^2 tokens 3.. do not matter
    j = 2
    k3, v3 = k.copy(), v.copy()
    for u in list(range(sink, j * block)) + list(range((j + 1) * block, n)) + list(range(n + j + 1, len(k))):
        k3[u] += 1.0
        v3[u] += 1.0
    o3, _ = oracle.sif_attend(q, k3, v3, n, block, sink, w.rope_base)
    np.testing.assert_allclose(o3[n + j], out[n + j], atol=1e-12, rtol=0)
    # ...but a token of its own block does
    v4 = v.copy()
    v4[j * block + 1] += 1.0
    o4, _ = oracle.sif_attend(q, k, v4, n, block, sink, w.rope_base)
    assert np.abs(o4[n + j] - out[n + j]).max() > 1e-3
