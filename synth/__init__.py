"""Seeded synthetic workloads for composed-KV attention.

This module only *generates inputs*: random K/V pools, kept-token index sets,
chunk orders, suffix Q/K/V, and (for int8 storage) the offline quantisation of
the pool.  It contains none of the arithmetic of the compose-and-attend path
(no RoPE, no position assignment, no attention), so both the float64 oracle and
the HIP path can consume the same arrays without sharing any of that code.

Workload shapes stand in for the paper's evaluation workloads, which are not
available here: documents of roughly 512 tokens reused with 4x compression
(Section 4.2), 16k-128k decode contexts (Section 4.3), roughly 4k-token
segments in 4k-64k contexts (Section 4.5).  No dataset content is used: every
value is drawn from N(0, 1).

Storage conventions (shared with the C ABI):
  * pool K/V      [rows][H_kv][D]; float32, bf16 (as uint16 bit patterns) or int8
  * pool scales   [rows][H_kv] float32 (int8 only), one for K and one for V
  * q             [B][S][H_q][D]  (float32 or bf16 bits), not yet RoPE-encoded
  * k_suf, v_suf  [B][S][H_kv][D]
  * segments      CSR over requests; each segment points at pool rows
                  [row0, row0 + span) and lists its kept indices (ascending).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

BASE_SEED = 2607_17715

# ---------------------------------------------------------------------------
# number formats (input generation only)
# ---------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even), as uint16 bits.

    Large arrays go through torch's float32 -> bfloat16 cast (also RNE; a CPU test
    checks the two agree), which is much faster than the integer form below."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.size >= (1 << 16):
        import torch
        return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return f32_to_bf16_bits_int(x)


def f32_to_bf16_bits_int(x: np.ndarray) -> np.ndarray:
    """Integer form of float32 -> bfloat16 RNE (the definition)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    out = (r >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def cast_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """float -> storage dtype ('f32' or 'bf16'); bf16 goes through fp32 (both RNE)."""
    x32 = np.asarray(x).astype(np.float32, copy=False)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(dtype)


def quantize_int8(x32: np.ndarray):
    """Offline symmetric int8 quantisation per (row, head) over the last axis.

    scale = max|x| / 127 in float32; q = clip(rint(x / scale), -127, 127) with the
    division in float64 and round-half-to-even.  Returns (int8 codes, f32 scales).
    """
    x32 = np.asarray(x32, dtype=np.float32)
    amax = np.max(np.abs(x32), axis=-1)
    scale = (amax / np.float32(127.0)).astype(np.float32)
    scale = np.where(scale == 0, np.float32(1.0), scale).astype(np.float32)
    qf = np.rint(x32.astype(np.float64) / scale[..., None].astype(np.float64))
    q = np.clip(qf, -127, 127).astype(np.int8)
    return q, scale


# ---------------------------------------------------------------------------
# workload container
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class Workload:
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_base: float
    pool_dtype: str              # 'f32' | 'bf16' | 'i8'
    act_dtype: str               # 'f32' | 'bf16'
    pool_k: np.ndarray
    pool_v: np.ndarray
    pool_k_scale: Optional[np.ndarray]
    pool_v_scale: Optional[np.ndarray]
    req_seg_off: np.ndarray      # int32 [B+1]
    seg_row0: np.ndarray         # int64 [n_seg]
    seg_span: np.ndarray         # int32 [n_seg]
    seg_orig_pos0: np.ndarray    # int32 [n_seg]
    seg_new_pos0: Optional[np.ndarray]  # int32 [n_seg] or None (accumulate)
    seg_kept_off: np.ndarray     # int32 [n_seg+1]
    kept_idx: np.ndarray         # int32 [total kept]
    suffix_len: int
    q: np.ndarray
    k_suf: np.ndarray
    v_suf: np.ndarray
    keys_pre_rope: bool = False  # pool keys taken as stored before RoPE (same values)
    pool_compressed: bool = False  # pool holds only kept rows, chunk by chunk

    @property
    def batch(self) -> int:
        return int(self.req_seg_off.shape[0] - 1)

    @property
    def n_segments(self) -> int:
        return int(self.seg_row0.shape[0])


@dataclasses.dataclass
class Spec:
    """Shape recipe of one synthetic workload."""
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_base: float
    pool_dtype: str
    act_dtype: str
    n_pool_chunks: int
    chunk_len: int
    prefix_len: int
    batch: int
    chunks_per_req: int
    order: str                   # 'natural' | 'shuffled' | 'draw'
    keep: tuple                  # ('count', m) | ('ratio', lo, hi) | ('c2', k) | ('all',)
    suffix_len: int
    layers: int = 1
    keys_pre_rope: bool = False


def spec(idx: int) -> Spec:
    """The synthetic workloads (1-based index): five prefill-style layers, then
    four decode steps."""
    if idx == 1:   # tiny fp32
        return Spec("tiny-fp32", 8, 2, 64, 1e4, "f32", "f32", 4, 256, 16, 1, 4,
                    "natural", ("count", 128), 32)
    if idx == 2:   # Llama-3-8B-shaped layer, bf16, shuffled chunk order
        return Spec("llama3-8b-layer-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 8, 512, 64,
                    1, 8, "shuffled", ("count", 128), 64)
    if idx == 3:   # batched ragged composition
        return Spec("ragged-batch-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 256, 512, 0,
                    16, 16, "draw", ("ratio", 0.1, 0.5), 128)
    if idx == 4:   # int8 storage, 32 layers
        return Spec("int8-32layer", 32, 8, 128, 5e5, "i8", "bf16", 64, 1024, 0, 1, 64,
                    "natural", ("count", 128), 32, layers=32)
    if idx == 5:   # 70B-shaped long suffix
        return Spec("70b-long-suffix-bf16", 64, 8, 128, 5e5, "bf16", "bf16", 32, 2048, 0,
                    1, 32, "natural", ("count", 1024), 2048)
    # decode steps (one new token) over a composed context of 2048-token chunks
    # with 4x / 16x compression or none, Llama-3-8B shapes
    if idx == 6:
        return Spec("decode-32k-4x-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 16, 2048, 0,
                    1, 16, "natural", ("count", 512), 1)
    if idx == 7:
        return Spec("decode-128k-4x-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 64, 2048, 0,
                    1, 64, "natural", ("count", 512), 1)
    if idx == 8:
        return Spec("decode-128k-16x-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 64, 2048, 0,
                    1, 64, "natural", ("count", 128), 1)
    if idx == 9:
        return Spec("decode-128k-1x-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 64, 2048, 0,
                    1, 64, "natural", ("all",), 1)
    # the Llama-3-8B layer with keys stored before RoPE, and with C^2-pattern kept
    # sets (block ends at compression 4)
    if idx == 10:
        return Spec("llama3-8b-layer-prerope-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 8, 512,
                    64, 1, 8, "shuffled", ("count", 128), 64, keys_pre_rope=True)
    if idx == 11:
        return Spec("llama3-8b-layer-c2x4-bf16", 32, 8, 128, 5e5, "bf16", "bf16", 8, 512, 64,
                    1, 8, "shuffled", ("c2", 4), 64)
    # the rest of the decode grid: contexts of 16k-128k tokens, uncompressed or
    # with 4x / 8x / 16x compression (Section 4.3)
    if 12 <= idx < 12 + len(DECODE_GRID):
        ctx, r = DECODE_GRID[idx - 12]
        return Spec(f"decode-{ctx}k-{r}x-bf16", 32, 8, 128, 5e5, "bf16", "bf16", ctx // 2, 2048,
                    0, 1, ctx // 2, "natural", ("all",) if r == 1 else ("count", 2048 // r), 1)
    raise ValueError(idx)


# (context in thousands of tokens, compression) of decode workloads 12 and on
DECODE_GRID = [(16, 1), (16, 4), (16, 8), (16, 16), (32, 1), (32, 8), (32, 16),
               (64, 1), (64, 4), (64, 8), (64, 16), (128, 8)]


def _kept_for_chunk(rng: np.random.Generator, keep: tuple, n: int) -> np.ndarray:
    kind = keep[0]
    if kind == "all":
        return np.arange(n, dtype=np.int32)
    if kind == "count":
        m = min(int(keep[1]), n)
    elif kind == "ratio":
        r = rng.uniform(keep[1], keep[2])
        m = max(1, int(np.floor(r * n)))
    elif kind == "c2":
        k = int(keep[1])
        m = -(-n // k)
        return np.array([min((j + 1) * k, n) - 1 for j in range(m)], dtype=np.int32)
    elif kind == "none":
        return np.zeros(0, dtype=np.int32)
    else:
        raise ValueError(kind)
    return np.sort(rng.choice(n, size=m, replace=False)).astype(np.int32)


def build(sp: Spec, layer: int = 0, seed: Optional[int] = None) -> Workload:
    """Draw one layer of a workload.  The layout (segments, kept sets, order) depends
    only on `seed`; tensors additionally on `layer`, so all layers share one plan."""
    seed = BASE_SEED if seed is None else seed
    ss = np.random.SeedSequence(seed)
    s_kept, s_order, s_ratio = [np.random.default_rng(s) for s in ss.spawn(3)]
    ts = np.random.SeedSequence([seed, 7919, layer])
    s_pk, s_pv, s_q, s_ks, s_vs, s_pre = [np.random.default_rng(s) for s in ts.spawn(6)]

    H, D, n, P = sp.n_kv_heads, sp.head_dim, sp.chunk_len, sp.prefix_len

    # pool values (prefix rows first, then chunk c at rows P + c*n)
    f32 = np.float32
    k0 = np.concatenate([s_pre.standard_normal((P, H, D), dtype=f32),
                          s_pk.standard_normal((sp.n_pool_chunks * n, H, D), dtype=f32)], axis=0)
    v0 = np.concatenate([s_pre.standard_normal((P, H, D), dtype=f32),
                          s_pv.standard_normal((sp.n_pool_chunks * n, H, D), dtype=f32)], axis=0)
    k_scale = v_scale = None
    if sp.pool_dtype == "i8":
        kb = bf16_bits_to_f32(cast_f64(k0, "bf16"))
        vb = bf16_bits_to_f32(cast_f64(v0, "bf16"))
        pool_k, k_scale = quantize_int8(kb)
        pool_v, v_scale = quantize_int8(vb)
    else:
        pool_k = cast_f64(k0, sp.pool_dtype)
        pool_v = cast_f64(v0, sp.pool_dtype)

    # per-chunk kept sets (one compressed form per chunk, shared by every use)
    keep_rng = s_ratio if sp.keep[0] == "ratio" else s_kept
    kept_sets = [_kept_for_chunk(keep_rng, sp.keep, n) for _ in range(sp.n_pool_chunks)]

    # which chunks each request composes, and in what order
    req_chunks = []
    for _ in range(sp.batch):
        if sp.order == "natural":
            ch = np.arange(sp.chunks_per_req)
        elif sp.order == "shuffled":
            ch = s_order.permutation(sp.chunks_per_req)
        elif sp.order == "draw":
            ch = s_order.choice(sp.n_pool_chunks, size=sp.chunks_per_req, replace=False)
        else:
            raise ValueError(sp.order)
        req_chunks.append([int(c) for c in ch])

    req_seg_off = [0]
    seg_row0, seg_span, seg_orig, kept_off, kept = [], [], [], [0], []
    for r in range(sp.batch):
        if P > 0:
            seg_row0.append(0); seg_span.append(P); seg_orig.append(0)
            kept.append(np.arange(P, dtype=np.int32)); kept_off.append(kept_off[-1] + P)
        for c in req_chunks[r]:
            seg_row0.append(P + c * n); seg_span.append(n); seg_orig.append(0)
            kept.append(kept_sets[c]); kept_off.append(kept_off[-1] + len(kept_sets[c]))
        req_seg_off.append(len(seg_row0))

    B, S = sp.batch, sp.suffix_len
    q = cast_f64(s_q.standard_normal((B, S, sp.n_q_heads, D)), sp.act_dtype)
    k_suf = cast_f64(s_ks.standard_normal((B, S, H, D)), sp.act_dtype)
    v_suf = cast_f64(s_vs.standard_normal((B, S, H, D)), sp.act_dtype)

    return Workload(
        name=sp.name, n_q_heads=sp.n_q_heads, n_kv_heads=H, head_dim=D,
        rope_base=sp.rope_base, pool_dtype=sp.pool_dtype, act_dtype=sp.act_dtype,
        pool_k=np.ascontiguousarray(pool_k), pool_v=np.ascontiguousarray(pool_v),
        pool_k_scale=k_scale, pool_v_scale=v_scale,
        req_seg_off=np.array(req_seg_off, np.int32),
        seg_row0=np.array(seg_row0, np.int64), seg_span=np.array(seg_span, np.int32),
        seg_orig_pos0=np.array(seg_orig, np.int32), seg_new_pos0=None,
        seg_kept_off=np.array(kept_off, np.int32),
        kept_idx=(np.concatenate(kept) if kept else np.zeros(0, np.int32)).astype(np.int32),
        suffix_len=S, q=q, k_suf=k_suf, v_suf=v_suf, keys_pre_rope=sp.keys_pre_rope)


def int8_layer_device(sp: Spec, layer: int, seed: int, device: str = "cuda") -> dict:
    """One layer of an int8-storage workload drawn straight on the device, for
    timing many layers without generating them on the host: pool K/V as N(0,1)
    rounded to bf16, then quantised per (row, head) as `quantize_int8` does
    (scale = max|x| / 127 in float32, codes rint(x / scale) with the division in
    float64, clipped to +-127); q, k_suf, v_suf as N(0,1) in bf16.  Seeded by
    (seed, layer) through torch's device generator, so the values differ from
    `build`'s numpy draws of the same layer while following the same recipe.
    The layout (rows, kept sets) is `build(sp, seed=seed)`'s: rows are indexed
    the same way.  Returns torch tensors k, v (int8), k_scale, v_scale (float32),
    q, k_suf, v_suf (bf16)."""
    import torch
    if sp.pool_dtype != "i8":
        raise ValueError("int8_layer_device draws int8-storage workloads only")
    states = np.random.SeedSequence([seed, 7919, layer, 2]).generate_state(5)
    gens = [torch.Generator(device=device) for _ in states]
    for g, st in zip(gens, states):
        g.manual_seed(int(st))
    rows = sp.prefix_len + sp.n_pool_chunks * sp.chunk_len
    H, D, B, S = sp.n_kv_heads, sp.head_dim, sp.batch, sp.suffix_len

    def normal_bf16(g, shape):
        return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)

    def quant(xb):
        x = xb.float()
        scale = x.abs().amax(dim=-1) / 127.0
        scale = torch.where(scale == 0, torch.ones_like(scale), scale)
        q = torch.round(x.double() / scale.double()[..., None]).clamp_(-127, 127).to(torch.int8)
        return q.contiguous(), scale.contiguous()

    k, k_scale = quant(normal_bf16(gens[0], (rows, H, D)))
    v, v_scale = quant(normal_bf16(gens[1], (rows, H, D)))
    return dict(k=k, v=v, k_scale=k_scale, v_scale=v_scale,
                q=normal_bf16(gens[2], (B, S, sp.n_q_heads, D)),
                k_suf=normal_bf16(gens[3], (B, S, H, D)),
                v_suf=normal_bf16(gens[4], (B, S, H, D)))


@dataclasses.dataclass
class SifWorkload:
    """Inputs of extraction-time SIF attention: `batch` sequences of n original
    tokens and their ceil(n / block) C^2 tokens, before RoPE."""
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_base: float
    act_dtype: str
    n_tokens: int
    block: int
    sink: int
    q: np.ndarray                # [B][L][H_q][d] in the act dtype's storage
    k: np.ndarray                # [B][L][H_kv][d]
    v: np.ndarray

    @property
    def batch(self) -> int:
        return int(self.q.shape[0])

    @property
    def seq_len(self) -> int:
        return int(self.q.shape[1])


def sif(name="sif", batch=2, n_tokens=300, block=4, sink=4, n_q_heads=8, n_kv_heads=2,
        head_dim=128, rope_base=5e5, act_dtype="bf16", seed=BASE_SEED + 100) -> SifWorkload:
    """Seeded N(0,1) queries, keys and values of SIF sequences."""
    L = n_tokens + -(-n_tokens // block)
    s_q, s_k, s_v = (np.random.Generator(np.random.PCG64(x))
                     for x in np.random.SeedSequence(seed).spawn(3))
    q = cast_f64(s_q.standard_normal((batch, L, n_q_heads, head_dim)), act_dtype)
    k = cast_f64(s_k.standard_normal((batch, L, n_kv_heads, head_dim)), act_dtype)
    v = cast_f64(s_v.standard_normal((batch, L, n_kv_heads, head_dim)), act_dtype)
    return SifWorkload(name, n_q_heads, n_kv_heads, head_dim, rope_base, act_dtype, n_tokens,
                       block, sink, q, k, v)


def sif_config(name: str) -> SifWorkload:
    """The SIF extraction workload of the benchmark: 16 Llama-3-8B-shaped document
    chunks of 512 tokens, one C^2 token per 4 (compression 4), a 4-token sink."""
    if name == "sif-extract-llama3-8b-bf16":
        return sif(name, batch=16, n_tokens=512, block=4, sink=4, n_q_heads=32, n_kv_heads=8,
                   head_dim=128, rope_base=5e5, act_dtype="bf16", seed=BASE_SEED + 12)
    raise ValueError(name)


def config(idx: int, layer: int = 0) -> Workload:
    """Workload `idx` (see spec), seeded with BASE_SEED + idx."""
    return build(spec(idx), layer=layer, seed=BASE_SEED + idx)


def small(pool_dtype="bf16", act_dtype=None, n_q_heads=8, n_kv_heads=2, head_dim=128,
          rope_base=5e5, n_pool_chunks=5, chunk_len=200, prefix_len=13, batch=2,
          chunks_per_req=3, order="draw", keep=("ratio", 0.1, 0.6), suffix_len=37,
          seed=12345, layer=0) -> Workload:
    """A small ragged workload for parity tests (several tiles and ragged tails)."""
    if act_dtype is None:
        act_dtype = "f32" if pool_dtype == "f32" else "bf16"
    sp = Spec("small", n_q_heads, n_kv_heads, head_dim, rope_base, pool_dtype, act_dtype,
              n_pool_chunks, chunk_len, prefix_len, batch, chunks_per_req, order, keep,
              suffix_len)
    return build(sp, layer=layer, seed=seed)


def compress_pool(w: Workload) -> Workload:
    """The same workload with its pool stored compressed: each distinct chunk
    (segment row0) keeps only its kept rows, in order, and segments point at
    their chunk's first kept row.  Values are copied, not redrawn, so results
    equal those of the full pool."""
    first_of = {}
    rows = []
    new_row0 = np.zeros_like(w.seg_row0)
    for c in range(w.n_segments):
        row0 = int(w.seg_row0[c])
        kept = w.kept_idx[w.seg_kept_off[c]:w.seg_kept_off[c + 1]].astype(np.int64)
        key = (row0, tuple(kept.tolist()))
        if key not in first_of:
            first_of[key] = sum(len(r) for r in rows)
            rows.append(row0 + kept)
        new_row0[c] = first_of[key]
    idx = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    take = lambda a: None if a is None else np.ascontiguousarray(a[idx])
    return dataclasses.replace(w, pool_k=take(w.pool_k), pool_v=take(w.pool_v),
                               pool_k_scale=take(w.pool_k_scale),
                               pool_v_scale=take(w.pool_v_scale), seg_row0=new_row0,
                               pool_compressed=True)


def with_overrides(w: Workload, **kw) -> Workload:
    return dataclasses.replace(w, **kw)
