"""Float64 oracle of the C2KV compose-and-attend path.

TEST INFRASTRUCTURE ONLY.  This is a plain, slow, obviously-correct statement
of what the compose-and-attend path computes.  Only `tests/`, the smoke check
and the benchmark's CPU-baseline leg use it.  It imports nothing from the HIP
library or its binding, and the product path must never call it.

Paper: "C2KV: Compressed and Composable KV Cache Reuse for Efficient LLM
Inference" (arXiv 2607.17715).  What is computed, step by step:

  1. decode storage exactly (fp32 / bf16 -> fp64; int8 * fp32 scale in fp64);
  2. lay the kept tokens of each reused segment out in request order and give
     each one its new position: offsets accumulate across segments, and a
     compressed segment keeps the span of its uncompressed tokens
     (Section 3.2, "Output and Reuse");
  3. re-rotate each cached key from its stored position to its new one
     (RoPE re-rotation, Appendix C; the Fixed-Pos ablation of Section 4.8 is
     the special case of no re-rotation);
  4. concatenate the segments as they are, with no blending or recompute
     (Section 3.2; Section 2.2, Eq. 3: KV_total = B(x_s, KV_1..KV_K));
  5. run the query tokens online over [KV_total, x_q] (Section 2.2, Eq. 4;
     Appendix D): standard softmax attention, grouped-query heads, causal
     among the query tokens.

Readings where the paper is silent (each is listed in the design notes):
  * stored keys are RoPE-encoded at their original positions orig_pos0 + j and
    are rotated by delta = new_pos0 - orig_pos0; this equals encoding the
    un-rotated key at the new position, because RoPE rotations compose;
  * RoPE uses theta_i = base^(-2i/d) with half-split pairing (i, i + d/2);
  * softmax scale 1/sqrt(d); query head h reads kv-head h // (H_q / H_kv);
  * suffix token t sits at position span_end + t, sees every composed slot and
    suffix tokens u <= t; span_end = the first position past every placed span
    (the maximum of new_pos0 + span over the request's segments: the end of the
    last span under accumulated placement, and of the furthest one when
    placements are given explicitly), since the query tokens run after the
    whole composed context (Section 2.2, Eq. 4);
  * lse is the natural-log log-sum-exp of the scaled scores.

Parity: pinned by the CPU tests (worked layout examples, RoPE group laws and
the complex-number form, equality with textbook causal attention through
torch SDPA, brute force on 2-token chunks, closed forms, row sums, exact int8
decode, permutation and split/merge invariance).
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np


# ---------------------------------------------------------------------------
# 1. storage decode (exact in float64)
# ---------------------------------------------------------------------------

def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64.  bf16 is the upper half of an
    IEEE binary32, so the value is exact."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def decode_storage(x: np.ndarray, dtype: str, scale: Optional[np.ndarray] = None
                   ) -> np.ndarray:
    """Stored K or V rows -> float64.

    'f32' and 'bf16' decode exactly.  'i8' multiplies each code by its
    per-(row, head) float32 scale; an 8-bit by 24-bit product fits in the 53-bit
    float64 significand, so that product is exact too."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return decode_bf16(x)
    if dtype == "i8":
        if scale is None:
            raise ValueError("int8 storage needs scales")
        return (np.asarray(x, dtype=np.int8).astype(np.float64)
                * np.asarray(scale, dtype=np.float32).astype(np.float64)[..., None])
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# rotary position embedding (the positional embedding the reused keys carry)
# ---------------------------------------------------------------------------

def rope_theta(d: int, base: float) -> np.ndarray:
    """theta_i = base^(-2i/d), i = 0 .. d/2-1, in float64."""
    i = np.arange(d // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * i / d)


def rope_rotate(x: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate the last axis of `x` (length d) to position(s) `pos`.

    Pair i is (x[i], x[i + d/2]); it turns by the angle pos * theta_i:
        x[i]       <- x[i] cos - x[i + d/2] sin
        x[i + d/2] <- x[i] sin + x[i + d/2] cos
    `pos` broadcasts against x.shape[:-1]; it may be negative (an inverse turn).
    """
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    h = d // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * rope_theta(d, base)
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


# ---------------------------------------------------------------------------
# 2. layout: kept-token slots and their new positions (Section 3.2)
# ---------------------------------------------------------------------------

def compose_layout(req_seg_off, seg_row0, seg_span, seg_orig_pos0, seg_kept_off,
                   kept_idx, seg_new_pos0=None, compressed: bool = False) -> dict:
    """Walk each request's segments in order and list its composed slots.

    Segment c of a request starts at new_pos0_c = sum of the spans of the
    segments before it (unless placements are given), so a compressed segment
    still advances the position by its full uncompressed span.  Its kept index j
    (ascending) becomes a slot with
        src_row = row0_c + j,  p_orig = orig_pos0_c + j,
        p_new   = new_pos0_c + j,  delta = new_pos0_c - orig_pos0_c.
    span_end of the request = the first position past every span: the maximum
    of new_pos0_c + span_c over its segments (with explicit placements the
    furthest span need not be the last segment's).  Spans are >= 1.
    Slot order = segments in request order, then kept indices ascending.
    compressed=True reads a pool that stores each chunk compressed (only its
    kept tokens, in order): the k-th kept token of a segment is row row0_c + k.
    """
    req_seg_off = np.asarray(req_seg_off, np.int64)
    B = len(req_seg_off) - 1
    out = {"src_row": [], "seg": [], "p_orig": [], "p_new": [], "delta": [],
           "span_end": np.zeros(B, np.int64), "composed_len": np.zeros(B, np.int64)}
    for r in range(B):
        pos = 0
        src, seg, po, pn, dl = [], [], [], [], []
        end = 0
        for c in range(int(req_seg_off[r]), int(req_seg_off[r + 1])):
            new0 = pos if seg_new_pos0 is None else int(seg_new_pos0[c])
            span = int(seg_span[c])
            row0 = int(seg_row0[c])
            orig0 = int(seg_orig_pos0[c])
            for k, j in enumerate(kept_idx[int(seg_kept_off[c]):int(seg_kept_off[c + 1])]):
                j = int(j)
                src.append(row0 + (k if compressed else j))
                seg.append(c)
                po.append(orig0 + j)
                pn.append(new0 + j)
                dl.append(new0 - orig0)
            pos = new0 + span
            end = max(end, new0 + span)
        out["src_row"].append(np.array(src, np.int64))
        out["seg"].append(np.array(seg, np.int64))
        out["p_orig"].append(np.array(po, np.int64))
        out["p_new"].append(np.array(pn, np.int64))
        out["delta"].append(np.array(dl, np.int64))
        out["span_end"][r] = end
        out["composed_len"][r] = len(src)
    return out


# ---------------------------------------------------------------------------
# 3 + 4. re-rotate and concatenate (Appendix C; Section 3.2)
# ---------------------------------------------------------------------------

def compose(layout: dict, pool_k, pool_v, pool_dtype: str, base: float,
            k_scale=None, v_scale=None, rerotate: bool = True, pre_rope: bool = False):
    """Composed cache of every request: list of (K [N_r, H_kv, d], V [N_r, H_kv, d]).

    Each slot's key is turned by its segment's delta (the same angle for all of
    its kv-heads); values are not rotated.  rerotate=False is the Fixed-Pos
    ablation (delta taken as 0).  pre_rope=True reads the stored keys as taken
    before positional encoding (Section 3.3.1) and encodes each one at its new
    position p_new instead."""
    res = []
    for r in range(len(layout["src_row"])):
        rows = layout["src_row"][r]
        k = decode_storage(pool_k[rows], pool_dtype,
                           None if k_scale is None else k_scale[rows])
        v = decode_storage(pool_v[rows], pool_dtype,
                           None if v_scale is None else v_scale[rows])
        if rerotate and len(rows):
            turn = layout["p_new" if pre_rope else "delta"][r].astype(np.float64)[:, None]
            turn = np.broadcast_to(turn, k.shape[:-1])              # the same for every head
            k = rope_rotate(k, turn, base)
        res.append((k, v))
    return res


# ---------------------------------------------------------------------------
# 5. attention of the query tokens over [KV_total, x_q] (Eq. 4; Appendix D)
# ---------------------------------------------------------------------------

def attend(k_cache, v_cache, q, k_suf, v_suf, span_end: int, base: float,
           scale: Optional[float] = None, rows: Optional[Sequence[int]] = None,
           return_probs: bool = False):
    """One request.  k_cache/v_cache [N, H_kv, d] (keys already at their final
    positions), q [S, H_q, d], k_suf/v_suf [S, H_kv, d] (not yet RoPE-encoded).

    Returns out [S', H_q, d] and lse [H_q, S'] for the selected suffix rows
    (all S by default), plus the probabilities [H_q, S', N + S] if asked.
    """
    q = np.asarray(q, np.float64)
    S, Hq, d = q.shape
    Hkv = k_suf.shape[1]
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else float(scale)
    t_all = np.arange(S)
    t_sel = t_all if rows is None else np.asarray(rows, np.int64)
    # suffix token t sits at position span_end + t
    q_rot = rope_rotate(q[t_sel], (span_end + t_sel)[:, None] * np.ones((1, Hq)), base)
    ks_rot = rope_rotate(np.asarray(k_suf, np.float64),
                         (span_end + t_all)[:, None] * np.ones((1, Hkv)), base)
    vs = np.asarray(v_suf, np.float64)
    kc = np.asarray(k_cache, np.float64).reshape(-1, Hkv, d)
    vc = np.asarray(v_cache, np.float64).reshape(-1, Hkv, d)
    N = kc.shape[0]
    out = np.zeros((len(t_sel), Hq, d))
    lse = np.zeros((Hq, len(t_sel)))
    probs = np.zeros((Hq, len(t_sel), N + S)) if return_probs else None
    visible = t_all[None, :] <= t_sel[:, None]            # [S', S] causal, inclusive
    for h in range(Hq):
        g = h // G
        keys = np.concatenate([kc[:, g, :], ks_rot[:, g, :]], axis=0)   # [N+S, d]
        vals = np.concatenate([vc[:, g, :], vs[:, g, :]], axis=0)
        s = scale * (q_rot[:, h, :] @ keys.T)                           # [S', N+S]
        s[:, N:] = np.where(visible, s[:, N:], -np.inf)
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        z = e.sum(axis=1, keepdims=True)
        p = e / z
        out[:, h, :] = p @ vals
        lse[h, :] = (m + np.log(z))[:, 0]
        if return_probs:
            probs[h] = p
    if return_probs:
        return out, lse, probs
    return out, lse


def compose_attend(w, rows: Optional[Sequence[int]] = None, requests=None,
                   rerotate: bool = True):
    """Whole path for a workload-like object `w` (attribute names of the C ABI's
    descriptor).  Returns (out [B][S'][H_q][d], lse [B][H_q][S'], layout)."""
    layout = compose_layout(w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0,
                            w.seg_kept_off, w.kept_idx, w.seg_new_pos0,
                            compressed=getattr(w, "pool_compressed", False))
    B = len(layout["src_row"])
    reqs = range(B) if requests is None else requests
    sub = {k: [layout[k][r] for r in reqs] if isinstance(layout[k], list) else layout[k]
           for k in layout}
    caches = compose(sub, w.pool_k, w.pool_v, w.pool_dtype, w.rope_base,
                     w.pool_k_scale, w.pool_v_scale, rerotate=rerotate,
                     pre_rope=getattr(w, "keys_pre_rope", False))
    act = w.act_dtype
    outs, lses = [], []
    for i, r in enumerate(reqs):
        kc, vc = caches[i]
        q = decode_storage(w.q[r], act)
        ks = decode_storage(w.k_suf[r], act)
        vs = decode_storage(w.v_suf[r], act)
        o, l = attend(kc, vc, q, ks, vs, int(layout["span_end"][r]), w.rope_base, rows=rows)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses), layout


# ---------------------------------------------------------------------------
# extraction-time attention with Structured Information Flow (Section 3.3)
# ---------------------------------------------------------------------------

def sif_positions(n: int, block: int) -> np.ndarray:
    """Positions of the sequence [x_1..x_n | c_1..c_m], m = ceil(n / block),
    0-based: original token t at t; C^2 token c_j (one per block of `block`
    originals) at the position of the last token of its block (Section 3.3.1)."""
    m = -(-n // block)
    j = np.arange(m)
    return np.concatenate([np.arange(n), np.minimum((j + 1) * block, n) - 1]).astype(np.int64)


def sif_mask(n: int, block: int, sink: int) -> np.ndarray:
    """visible[t, u] over the same sequence (Section 3.3.2): an original token
    sees the originals up to itself and no C^2 token; C^2 token c_j sees the
    originals of its block B(j) and of the sink block B(0) (here the first `sink`
    originals) and the C^2 tokens c_1..c_j."""
    m = -(-n // block)
    L = n + m
    vis = np.zeros((L, L), bool)
    for t in range(n):
        vis[t, :t + 1] = True
    for j in range(m):
        row = n + j
        vis[row, j * block:min((j + 1) * block, n)] = True
        vis[row, :sink] = True
        vis[row, n:n + j + 1] = True
    return vis


def sif_attend(q, k, v, n: int, block: int, sink: int, base: float,
               scale: Optional[float] = None):
    """One sequence of n originals and their C^2 tokens.  q [L, H_q, d],
    k, v [L, H_kv, d] before RoPE, L = n + ceil(n / block).  Returns
    out [L, H_q, d] and lse [H_q, L]."""
    q = np.asarray(q, np.float64)
    L, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else float(scale)
    pos = sif_positions(n, block)
    assert len(pos) == L
    q_rot = rope_rotate(q, pos[:, None] * np.ones((1, Hq)), base)
    k_rot = rope_rotate(np.asarray(k, np.float64), pos[:, None] * np.ones((1, Hkv)), base)
    vals = np.asarray(v, np.float64)
    vis = sif_mask(n, block, sink)
    out = np.zeros((L, Hq, d))
    lse = np.zeros((Hq, L))
    for h in range(Hq):
        g = h // G
        s = scale * (q_rot[:, h, :] @ k_rot[:, g, :].T)
        s = np.where(vis, s, -np.inf)
        mx = s.max(axis=1, keepdims=True)
        e = np.exp(s - mx)
        z = e.sum(axis=1, keepdims=True)
        out[:, h, :] = (e / z) @ vals[:, g, :]
        lse[h, :] = (mx + np.log(z))[:, 0]
    return out, lse


# ---------------------------------------------------------------------------
# combining attention over a partition of the keys
# ---------------------------------------------------------------------------

def merge_partials(parts):
    """Combine (out_i, lse_i) computed over disjoint key subsets of the same
    query rows: lse = log sum_i exp(lse_i); out = sum_i exp(lse_i - lse) out_i.
    out_i [..., d], lse_i [...] (same leading shape)."""
    lses = np.stack([np.asarray(l, np.float64) for _, l in parts])
    outs = np.stack([np.asarray(o, np.float64) for o, _ in parts])
    m = lses.max(axis=0)
    w = np.exp(lses - m)
    z = w.sum(axis=0)
    lse = m + np.log(z)
    out = (w[..., None] * outs).sum(axis=0) / z[..., None]
    return out, lse
