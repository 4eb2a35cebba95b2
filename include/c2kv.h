/*
 * c2kv.h — C ABI of the C2KV compose-and-attend path on MI355X (gfx950).
 *
 * Paper: "C2KV: Compressed and Composable KV Cache Reuse for Efficient LLM
 * Inference" (arXiv 2607.17715).  The two-stage reuse problem of Section 2.2
 * (Eq. 2-4) maps onto this interface as follows:
 *   - KV_reuse_k (Eq. 2), the stored per-document caches   -> a `c2kv_pool` of
 *     token rows plus, per placed segment, its kept-token index set;
 *   - the static context x_s                               -> an ordinary
 *     segment with every token kept, placed first;
 *   - the blender B (Eq. 3): retrieve, give new positions, concatenate
 *     (Section 3.2 "Output and Reuse"; Appendix C)         -> `c2kv_compose`;
 *   - the attention of F over [KV_total, x_q] (Eq. 4)      -> `c2kv_attend`;
 *   - both at once, without materialising KV_total         -> `c2kv_compose_attend`.
 *
 * Typical use (one batch of requests; every layer reuses the plan, since the
 * kept sets and positions are the same for all layers and heads):
 *   c2kv_plan_create(&cfg, &desc, suffix_len, NULL, &plan);          host, once
 *   c2kv_plan_get_info(plan, &info);             workspace_bytes, n_pages, ...
 *   c2kv_plan_upload(plan, workspace, info.workspace_bytes, stream); once
 *   per layer, either
 *     c2kv_compose_attend(plan, &pool, q, k_suf, v_suf, out, lse, stream);
 *   or, keeping the composed cache (decode steps attend to it again):
 *     c2kv_compose(plan, &pool, k_pages, v_pages, NULL, NULL, NULL, stream);
 *     c2kv_attend(plan, k_pages, v_pages, q, k_suf, v_suf, out, lse, stream);
 *   c2kv_plan_destroy(plan);
 *
 * Conventions shared by every call
 *   Ownership.  The caller owns every buffer.  The library never allocates
 *     device memory: scratch lives in a caller-provided workspace whose size
 *     `c2kv_plan_get_info` reports.  A plan is a host object owned by the caller.
 *   Pointers.  Arrays in `c2kv_compose_desc` are HOST pointers, read only during
 *     `c2kv_plan_create`.  Every other data pointer is a DEVICE pointer.
 *   Streams.  `stream` is a hipStream_t (NULL = the null stream).  Device work is
 *     enqueued asynchronously on it; no call synchronises the device.  Calls that
 *     share one plan (and so one workspace) must be ordered on one stream.
 *   Errors.  Every call returns a c2kv_status and never aborts; the text of the
 *     last error on the calling thread is available from `c2kv_last_error`.
 *     C2KV_E_INVAL       bad argument (null pointer, shape, index, ordering);
 *     C2KV_E_UNSUPPORTED valid but not built (e.g. head_dim 96, int8 with f32 acts);
 *     C2KV_E_WORKSPACE   workspace missing or too small;
 *     C2KV_E_STATE       plan not uploaded to a workspace;
 *     C2KV_E_HIP         a HIP runtime or launch error (message has the HIP text);
 *     C2KV_E_NOMEM       host allocation failed.
 *
 * Layouts (row-major, innermost last)
 *   pool K/V        [n_rows][H_kv][D]          storage dtype (F32, BF16 or I8)
 *   pool scales     [n_rows][H_kv] float32     I8 only: x = code * scale, per
 *                                              (token, kv-head), separate for K and V
 *   q               [B][S][H_q][D]   act dtype, not yet RoPE-encoded
 *   k_suf, v_suf    [B][S][H_kv][D]  act dtype, k_suf not yet RoPE-encoded
 *   out             [B][S][H_q][D]   act dtype
 *   lse             [B][H_q][S]      float32, natural-log log-sum-exp (optional)
 *   k_pages         [n_pages][H_kv][page_size][D]   act dtype, keys at final positions
 *   v_pages         [n_pages][H_kv][D][page_size]   act dtype, values, TRANSPOSED in a page
 *   A request's composed slot s lives in page block_table[b][s / page_size] at
 *   offset s % page_size; a request's pages are consecutive
 *   (block_table[b][i] = block_table[b][0] + i).
 *
 * Semantics (the readings of the paper this library implements)
 *   - Stored keys carry RoPE at their original positions orig_pos0 + j; compose
 *     turns them by delta = new_pos0 - orig_pos0 (RoPE re-rotation, Appendix C).
 *   - Placement is span-preserving (Section 3.2): unless given explicitly,
 *     new_pos0 of a segment = sum of the uncompressed spans before it in its
 *     request; kept index j lands at new_pos0 + j.
 *   - Composed slot order = segments in request order, kept indices ascending.
 *   - RoPE: theta_i = base^(-2i/D), pairs (i, i + D/2).  Softmax scale 1/sqrt(D)
 *     unless given.  Query head h reads kv-head h / (H_q / H_kv).
 *   - Suffix token t is at position span_end + t, where span_end is the first
 *     position past every placed span: the maximum over the request's segments
 *     of new_pos0 + seg_span (with accumulated placement, the end of the last
 *     segment's span; with explicit placements, whichever span reaches
 *     furthest, which need not be the last segment's).  The query tokens run
 *     after the whole composed context (Section 2.2, Eq. 4).  Suffix token t
 *     sees every composed slot and suffix tokens u <= t.
 */
#ifndef C2KV_H
#define C2KV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum c2kv_status {
  C2KV_OK = 0,
  C2KV_E_INVAL = -1,
  C2KV_E_UNSUPPORTED = -2,
  C2KV_E_WORKSPACE = -3,
  C2KV_E_HIP = -4,
  C2KV_E_NOMEM = -5,
  C2KV_E_STATE = -6
} c2kv_status;

typedef enum c2kv_dtype { C2KV_F32 = 0, C2KV_BF16 = 1, C2KV_I8 = 2 } c2kv_dtype;

/* Per-layer attention shape (Section 2.1, Eq. 1: the per-layer cache). */
typedef struct c2kv_attn_cfg {
  int32_t n_q_heads;      /* H_q, a multiple of n_kv_heads                         */
  int32_t n_kv_heads;     /* H_kv                                                  */
  int32_t head_dim;       /* D: 64 or 128                                          */
  c2kv_dtype act_dtype;   /* F32 or BF16: q, k_suf, v_suf, out and the pages       */
  double rope_base;       /* > 0                                                   */
  float softmax_scale;    /* <= 0 selects 1/sqrt(D)                                */
} c2kv_attn_cfg;

/* The composition B(x_s, KV_1..KV_K) of a batch of requests (Section 2.2, Eq. 3;
 * Section 3.2).  HOST arrays, read only inside c2kv_plan_create. */
/* How the pool stores its keys. */
typedef enum c2kv_key_encoding {
  C2KV_KEYS_ROPE_AT_ORIG = 0,   /* RoPE-encoded at seg_orig_pos0 + j; composing turns each
                                   key by delta = new_pos0 - orig_pos0 (Section 3.2
                                   "Output and Reuse", Appendix C)                        */
  C2KV_KEYS_PRE_ROPE = 1        /* stored before positional encoding (Section 3.3.1);
                                   composing encodes each key at its new position
                                   new_pos0 + j.  The cos/sin table then has one row per
                                   composed slot instead of one per segment               */
} c2kv_key_encoding;

/* Where a segment's kept tokens sit in the pool. */
typedef enum c2kv_pool_layout {
  C2KV_POOL_FULL = 0,         /* chunks stored whole: kept token j of a segment is pool
                                 row seg_row0 + j                                       */
  C2KV_POOL_COMPRESSED = 1    /* chunks stored compressed, only their kept tokens, in
                                 order (Section 3.2: the compressed cache is what is
                                 saved): the k-th kept token of a segment is pool row
                                 seg_row0 + k; its position still comes from kept_idx */
} c2kv_pool_layout;

typedef struct c2kv_compose_desc {
  int32_t batch;                 /* B >= 1                                          */
  int32_t n_segments;            /* total segments over all requests                */
  const int32_t* req_seg_off;    /* [B+1] CSR: segments of request b are
                                    req_seg_off[b] .. req_seg_off[b+1]-1, in order  */
  const int64_t* seg_row0;       /* [n_segments] pool row of the segment's token 0  */
  const int32_t* seg_span;       /* [n_segments] uncompressed length n (>= 1;
                                    C2KV_E_INVAL otherwise)                         */
  const int32_t* seg_orig_pos0;  /* [n_segments] position token 0 was encoded at    */
  const int32_t* seg_new_pos0;   /* [n_segments] placement, or NULL: span-preserving
                                    accumulation from 0 within each request         */
  const int32_t* seg_kept_off;   /* [n_segments+1] CSR into kept_idx                */
  const int32_t* kept_idx;       /* strictly ascending within a segment, each in
                                    [0, seg_span); a segment may keep nothing       */
  int32_t key_encoding;          /* c2kv_key_encoding of the pool's keys            */
  int32_t pool_layout;           /* c2kv_pool_layout                                */
} c2kv_compose_desc;

/* Launch-shape options.  Zero fields select the defaults. */
typedef struct c2kv_plan_opts {
  int32_t page_size;       /* tokens per page, a multiple of 64 (default 64)       */
  int32_t kv_splits;       /* > 0: key splits per row block (default: automatic)   */
  int32_t rows_per_block;  /* 64, 128 or 256 query rows per workgroup; automatic:
                              256 when a (request, kv-head) has at least 256
                              query rows (S * H_q / H_kv), else 128 (bf16, more
                              than 64 rows) or 64                               */
  int32_t num_cus;         /* compute units to size the work list for (256)       */
  int32_t merge_mode;      /* combining key splits: 0 automatic (currently the
                              separate kernel), 1 the last split of a row block
                              merges inside the attention kernel, 2 a separate
                              merge kernel                                        */
} c2kv_plan_opts;

/* The stored caches KV_reuse (Section 2.2, Eq. 2): device memory, caller-owned. */
typedef struct c2kv_pool {
  c2kv_dtype dtype;        /* storage dtype: F32, BF16 or I8                       */
  const void* k;           /* [n_rows][H_kv][D]                                    */
  const void* v;           /* [n_rows][H_kv][D]                                    */
  const float* k_scale;    /* [n_rows][H_kv], I8 only (else NULL)                  */
  const float* v_scale;    /* [n_rows][H_kv], I8 only (else NULL)                  */
  int64_t n_rows;
} c2kv_pool;

typedef struct c2kv_plan c2kv_plan;

typedef struct c2kv_plan_info {
  int32_t batch;
  int32_t suffix_len;
  int32_t page_size;
  int32_t n_pages;           /* pages the composed cache needs in total           */
  int32_t max_pages;         /* columns of the block table                        */
  int32_t n_segments;
  int64_t total_slots;       /* sum over requests of composed length              */
  int64_t max_src_row;       /* largest pool row any slot reads (-1 if none)      */
  size_t workspace_bytes;    /* device workspace c2kv_plan_upload needs           */
  int32_t rows_per_block;
  int32_t n_work_items;      /* attention workgroups per call                     */
  int32_t n_merge_groups;    /* row blocks whose key splits need merging          */
  int32_t max_splits;
} c2kv_plan_info;

/* Build the host plan (Section 3.2 placement; the layout is a pure function of
 * desc).  Validates desc: C2KV_E_INVAL on bad CSR offsets, kept indices not
 * strictly ascending or outside [0, span), negative rows, positions or deltas
 * outside int32, suffix_len < 1, unsupported shapes.  *out is set only on OK. */
c2kv_status c2kv_plan_create(const c2kv_attn_cfg* cfg, const c2kv_compose_desc* desc,
                             int32_t suffix_len, const c2kv_plan_opts* opts,
                             c2kv_plan** out);
void c2kv_plan_destroy(c2kv_plan* plan);

c2kv_status c2kv_plan_get_info(const c2kv_plan* plan, c2kv_plan_info* info);

/* Host copies of the layout.  composed_len, span_end: [B].  src_row, p_new,
 * delta: [total_slots] in slot order (any may be NULL).  block_table:
 * [B][max_pages], unused entries -1. */
c2kv_status c2kv_plan_get_requests(const c2kv_plan* plan, int32_t* composed_len,
                                   int32_t* span_end);
c2kv_status c2kv_plan_get_slots(const c2kv_plan* plan, int64_t* src_row, int32_t* p_new,
                                int32_t* delta);
c2kv_status c2kv_plan_get_block_table(const c2kv_plan* plan, int32_t* block_table);

/* Copy the plan's tables (slot table, cos/sin of every delta and suffix position
 * computed in float64, block table, work list) into `workspace` (device memory,
 * 256-byte aligned, at least workspace_bytes) on `stream`, and bind the plan to
 * it.  The plan must outlive every call that uses it. */
c2kv_status c2kv_plan_upload(c2kv_plan* plan, void* workspace, size_t workspace_bytes,
                             void* stream);

/* Blender B (Eq. 3): gather each request's kept rows from the pool, decode them
 * (I8: code * scale in fp32), turn keys by their segment's delta, and write the
 * composed cache into pages (act dtype; F32 acts need an F32 pool).
 * Optional device outputs (NULL to skip): slot_src_row [total_slots] int64,
 * slot_pos [total_slots] int32 (new positions), block_table [B][max_pages] int32.
 * Pool rows read must be < pool->n_rows (C2KV_E_INVAL otherwise). */
c2kv_status c2kv_compose(const c2kv_plan* plan, const c2kv_pool* pool, void* k_pages,
                         void* v_pages, int64_t* slot_src_row, int32_t* slot_pos,
                         int32_t* block_table, void* stream);

/* F's attention (Eq. 4) over a composed paged cache written by c2kv_compose with
 * this plan: suffix q and k_suf get RoPE at span_end + t, then every query head
 * attends to all composed slots and the causal suffix.  lse may be NULL. */
c2kv_status c2kv_attend(const c2kv_plan* plan, const void* k_pages, const void* v_pages,
                        const void* q, const void* k_suf, const void* v_suf, void* out,
                        float* lse, void* stream);

/* compose + attend in one pass: the kept rows are gathered, decoded and turned
 * while they are loaded for attention, and the composed cache is never written.
 * Same result as c2kv_compose followed by c2kv_attend, bit for bit (both round a
 * turned key once to the act dtype and use the same arithmetic after). */
c2kv_status c2kv_compose_attend(const c2kv_plan* plan, const c2kv_pool* pool,
                                const void* q, const void* k_suf, const void* v_suf,
                                void* out, float* lse, void* stream);

/* Bytes of the static scratch array that c2kv_compose_attend_static uses on each
 * GPU (held from the library's load until the process ends). */
#define C2KV_STATIC_SCRATCH_BYTES (32u << 20)

/* For callers that cannot allocate device memory or bind a workspace: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * same computation as c2kv_compose_attend, bit for bit (the same kernels), but
 * the plan's tables and the key-split partials live in a static device array of
 * C2KV_STATIC_SCRATCH_BYTES on the current GPU instead of a caller workspace; the
 * plan need not be uploaded.  The call copies the plan's tables into the array
 * on `stream` (which must belong to the current GPU), then launches.  It calls
 * no hipMalloc, hipFree or other allocating routine.
 *   C2KV_E_WORKSPACE  the plan's workspace_bytes exceed C2KV_STATIC_SCRATCH_BYTES
 *                     (checked before any device work);
 *   otherwise the errors of c2kv_compose_attend.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (other streams, other threads) race
 * and must be ordered by the caller. */
c2kv_status c2kv_compose_attend_static(const c2kv_plan* plan, const c2kv_pool* pool,
                                       const void* q, const void* k_suf, const void* v_suf,
                                       void* out, float* lse, void* stream);

/* Extraction-time attention with Structured Information Flow (Section 3.3):
 * each of `batch` sequences holds n_tokens original tokens followed by one C^2
 * token per block of `block` originals, m = ceil(n_tokens / block) of them.  The
 * plan is used with c2kv_plan_upload and c2kv_attend (k_pages = v_pages = NULL):
 * q [batch][n+m][H_q][D], k_suf and v_suf [batch][n+m][H_kv][D] (all tokens,
 * before RoPE), out [batch][n+m][H_q][D], lse [batch][H_q][n+m].  RoPE puts
 * original token t at position t and C^2 token j at the position of the last
 * token of its block, min((j+1) block, n) - 1.  The mask (Section 3.3.2):
 * originals attend causally to originals only; C^2 token j attends to the
 * originals of its block, to the first `sink` originals (the sink block B(0),
 * whose size the paper leaves open), and to C^2 tokens 0..j.  C2KV_E_INVAL for
 * batch, n_tokens or block < 1, or sink outside [0, n_tokens]. */
c2kv_status c2kv_sif_plan_create(const c2kv_attn_cfg* cfg, int32_t batch, int32_t n_tokens,
                                 int32_t block, int32_t sink, const c2kv_plan_opts* opts,
                                 c2kv_plan** out);

/* The load step (Appendix C: compressed caches move to the GPU before they are
 * repositioned).  Page-locked host memory that kernels can also read in place:
 * *host is its CPU address, *device the address to put in a c2kv_pool for
 * reads over the host link (zero-copy).  Free with c2kv_host_free(host).
 * C2KV_E_HIP if the runtime cannot provide it. */
c2kv_status c2kv_host_alloc(size_t bytes, void** host, void** device);
c2kv_status c2kv_host_free(void* host);

/* Copy engines instead of zero-copy reads: for every segment of the plan the
 * pool rows its kept tokens read (first to last; with a compressed pool exactly
 * its kept rows; ranges of neighbouring segments merged) are copied from `src`
 * to the same rows of `dst`, K and V (and the int8 scales), with asynchronous
 * copies on `stream`.  src may be host (c2kv_host_alloc) or device memory; dst
 * is a device pool of the same dtype with n_rows covering the plan.  Returns
 * C2KV_E_INVAL on mismatched pools. */
c2kv_status c2kv_load(const c2kv_plan* plan, const c2kv_pool* src, const c2kv_pool* dst,
                      void* stream);

/* Per-kernel timing for measurement: when enabled, every kernel is launched
 * with a pair of HIP events that its dispatch stamps at kernel start and end
 * (on the kernel's own stream).  c2kv_timing_read synchronises on them and
 * returns the summed milliseconds and launch count of kernel `name`
 * ("compose", "attn_paged", "attn_pool", "merge") since the last reset.
 * Launches with timing on are not meant for graph capture. */
c2kv_status c2kv_timing_enable(int32_t on);
c2kv_status c2kv_timing_reset(void);
c2kv_status c2kv_timing_read(const char* name, double* total_ms, int64_t* launches);

const char* c2kv_last_error(void);
const char* c2kv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* C2KV_H */
