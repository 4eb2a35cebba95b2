// C ABI of the compose-and-attend path (declared in include/c2kv.h): argument
// checks, workspace binding, kernel launches on the caller's stream, optional
// per-kernel event timing, and the thread-local error text.
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "c2kv.h"
#include "launch.hpp"
#include "plan.hpp"

namespace {

thread_local std::string g_last_error;

c2kv_status fail(c2kv_status st, std::string msg) {
  g_last_error = std::move(msg);
  return st;
}

c2kv_status hip_fail(hipError_t e, const char* what) {
  return fail(C2KV_E_HIP, std::string(what) + ": " + hipGetErrorName(e) + " (" +
                              hipGetErrorString(e) + ")");
}

// ---- optional per-kernel timing --------------------------------------------
struct Timing {
  std::mutex mu;
  bool on = false;
  struct Rec { hipEvent_t a, b; };
  std::map<std::string, std::vector<Rec>> recs;
  std::vector<hipEvent_t> spare;
};
Timing g_timing;

hipEvent_t take_event() {
  if (!g_timing.spare.empty()) {
    hipEvent_t e = g_timing.spare.back();
    g_timing.spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Runs `launch(ev0, ev1)`; when timing is on, the events (stamped by the
// kernel's own dispatch at its start and end) are filed under `name`.
template <typename F>
hipError_t timed(const char* name, F&& launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    on = g_timing.on;
  }
  if (!on) return launch(nullptr, nullptr);
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    a = take_event();
    b = take_event();
  }
  hipError_t e = a && b ? launch(a, b) : hipErrorOutOfMemory;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (e != hipSuccess) {
    // events of a launch that did not happen go back to the spare list
    if (a) g_timing.spare.push_back(a);
    if (b) g_timing.spare.push_back(b);
    return e;
  }
  g_timing.recs[name].push_back({a, b});
  return hipSuccess;
}

bool check_plan(const c2kv_plan* plan, c2kv_status* st) {
  if (!plan) { *st = fail(C2KV_E_INVAL, "plan is NULL"); return false; }
  if (!plan->p.d_workspace) {
    *st = fail(C2KV_E_STATE, "plan is not uploaded (call c2kv_plan_upload first)");
    return false;
  }
  return true;
}

bool check_pool(const c2kv::Plan& p, const c2kv_pool* pool, c2kv_status* st) {
  if (!pool || !pool->k || !pool->v) {
    *st = fail(C2KV_E_INVAL, "pool or its K/V pointer is NULL");
    return false;
  }
  if (pool->dtype != C2KV_F32 && pool->dtype != C2KV_BF16 && pool->dtype != C2KV_I8) {
    *st = fail(C2KV_E_INVAL, "pool dtype must be F32, BF16 or I8");
    return false;
  }
  const bool ok_combo = (pool->dtype == C2KV_F32 && p.cfg.act_dtype == C2KV_F32) ||
                        (pool->dtype == C2KV_BF16 && p.cfg.act_dtype == C2KV_BF16) ||
                        (pool->dtype == C2KV_I8 && p.cfg.act_dtype == C2KV_BF16);
  if (!ok_combo) {
    *st = fail(C2KV_E_UNSUPPORTED,
               "pool/act dtype combination not built (F32/F32, BF16/BF16, I8/BF16)");
    return false;
  }
  if (pool->dtype == C2KV_I8 && (!pool->k_scale || !pool->v_scale)) {
    *st = fail(C2KV_E_INVAL, "I8 pool needs k_scale and v_scale");
    return false;
  }
  if (p.max_src_row >= pool->n_rows) {
    *st = fail(C2KV_E_INVAL, "a kept token reads pool row " + std::to_string(p.max_src_row) +
                                 " but the pool has " + std::to_string(pool->n_rows) + " rows");
    return false;
  }
  return true;
}

bool check_io(const void* q, const void* ks, const void* vs, const void* out,
              c2kv_status* st) {
  if (!q || !ks || !vs || !out) {
    *st = fail(C2KV_E_INVAL, "q, k_suf, v_suf and out must not be NULL");
    return false;
  }
  return true;
}

}  // namespace

extern "C" {

const char* c2kv_last_error(void) { return g_last_error.c_str(); }

const char* c2kv_version(void) { return "c2kv 0.1.0 gfx950"; }

c2kv_status c2kv_plan_create(const c2kv_attn_cfg* cfg, const c2kv_compose_desc* desc,
                             int32_t suffix_len, const c2kv_plan_opts* opts,
                             c2kv_plan** out) {
  if (!cfg || !desc || !out) return fail(C2KV_E_INVAL, "cfg, desc and out must not be NULL");
  c2kv_plan* plan = new (std::nothrow) c2kv_plan;
  if (!plan) return fail(C2KV_E_NOMEM, "cannot allocate plan");
  std::string err;
  c2kv_status st;
  try {
    st = c2kv::build_plan(*cfg, *desc, suffix_len, opts, plan->p, err);
  } catch (const std::bad_alloc&) {
    st = C2KV_E_NOMEM;
    err = "host allocation failed while building the plan";
  }
  if (st != C2KV_OK) {
    delete plan;
    return fail(st, err);
  }
  *out = plan;
  return C2KV_OK;
}

c2kv_status c2kv_sif_plan_create(const c2kv_attn_cfg* cfg, int32_t batch, int32_t n_tokens,
                                 int32_t block, int32_t sink, const c2kv_plan_opts* opts,
                                 c2kv_plan** out) {
  if (!cfg || !out) return fail(C2KV_E_INVAL, "cfg and out must not be NULL");
  c2kv_plan* plan = new (std::nothrow) c2kv_plan;
  if (!plan) return fail(C2KV_E_NOMEM, "cannot allocate plan");
  std::string err;
  c2kv_status st;
  try {
    st = c2kv::build_sif_plan(*cfg, batch, n_tokens, block, sink, opts, plan->p, err);
  } catch (const std::bad_alloc&) {
    st = C2KV_E_NOMEM;
    err = "host allocation failed while building the plan";
  }
  if (st != C2KV_OK) {
    delete plan;
    return fail(st, err);
  }
  *out = plan;
  return C2KV_OK;
}

void c2kv_plan_destroy(c2kv_plan* plan) { delete plan; }

c2kv_status c2kv_plan_get_info(const c2kv_plan* plan, c2kv_plan_info* info) {
  if (!plan || !info) return fail(C2KV_E_INVAL, "plan and info must not be NULL");
  const c2kv::Plan& p = plan->p;
  info->batch = p.batch;
  info->suffix_len = p.suffix_len;
  info->page_size = p.page_size;
  info->n_pages = p.n_pages;
  info->max_pages = p.max_pages;
  info->n_segments = p.n_segments;
  info->total_slots = static_cast<int64_t>(p.slot_src.size());
  info->max_src_row = p.max_src_row;
  info->workspace_bytes = p.ws.total;
  info->rows_per_block = p.rows_per_block;
  info->n_work_items = static_cast<int32_t>(p.items.size());
  info->n_merge_groups = static_cast<int32_t>(p.merges.size());
  info->max_splits = p.max_splits;
  return C2KV_OK;
}

c2kv_status c2kv_plan_get_requests(const c2kv_plan* plan, int32_t* composed_len,
                                   int32_t* span_end) {
  if (!plan) return fail(C2KV_E_INVAL, "plan is NULL");
  const c2kv::Plan& p = plan->p;
  for (int b = 0; b < p.batch; ++b) {
    if (composed_len) composed_len[b] = p.req_slot0[b + 1] - p.req_slot0[b];
    if (span_end) span_end[b] = p.span_end[b];
  }
  return C2KV_OK;
}

c2kv_status c2kv_plan_get_slots(const c2kv_plan* plan, int64_t* src_row, int32_t* p_new,
                                int32_t* delta) {
  if (!plan) return fail(C2KV_E_INVAL, "plan is NULL");
  const c2kv::Plan& p = plan->p;
  const size_t n = p.slot_src.size();
  for (size_t i = 0; i < n; ++i) {
    if (src_row) src_row[i] = p.slot_src[i];
    if (p_new) p_new[i] = p.slot_pos[i];
    if (delta) delta[i] = p.slot_delta[i];
  }
  return C2KV_OK;
}

c2kv_status c2kv_plan_get_block_table(const c2kv_plan* plan, int32_t* block_table) {
  if (!plan || !block_table) return fail(C2KV_E_INVAL, "plan and block_table must not be NULL");
  std::memcpy(block_table, plan->p.block_table.data(),
              plan->p.block_table.size() * sizeof(int32_t));
  return C2KV_OK;
}

c2kv_status c2kv_plan_upload(c2kv_plan* plan, void* workspace, size_t workspace_bytes,
                             void* stream) {
  if (!plan) return fail(C2KV_E_INVAL, "plan is NULL");
  c2kv::Plan& p = plan->p;
  if (!workspace) return fail(C2KV_E_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(C2KV_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < p.ws.total)
    return fail(C2KV_E_WORKSPACE, "workspace has " + std::to_string(workspace_bytes) +
                                      " bytes, plan needs " + std::to_string(p.ws.total));
  hipError_t e = hipMemcpyAsync(workspace, p.image.data(), p.image.size(),
                                hipMemcpyHostToDevice, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (plan upload)");
  p.d_workspace = workspace;
  p.d_workspace_bytes = workspace_bytes;
  return C2KV_OK;
}

c2kv_status c2kv_compose(const c2kv_plan* plan, const c2kv_pool* pool, void* k_pages,
                         void* v_pages, int64_t* slot_src_row, int32_t* slot_pos,
                         int32_t* block_table, void* stream) {
  c2kv_status st;
  if (!check_plan(plan, &st)) return st;
  const c2kv::Plan& p = plan->p;
  if (!check_pool(p, pool, &st)) return st;
  if ((!k_pages || !v_pages) && p.n_pages > 0)
    return fail(C2KV_E_INVAL, "k_pages and v_pages must not be NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = timed("compose", [&](hipEvent_t e0, hipEvent_t e1) {
    return c2kv::launch_compose(p, p.d_workspace, pool->dtype, pool->k, pool->v, pool->k_scale,
                                pool->v_scale, k_pages, v_pages, slot_src_row, slot_pos, s, e0, e1);
  });
  if (e != hipSuccess) return hip_fail(e, "compose launch");
  if (block_table) {
    e = hipMemcpyAsync(block_table,
                       static_cast<const uint8_t*>(p.d_workspace) + p.ws.block_table,
                       p.block_table.size() * sizeof(int32_t), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (block table)");
  }
  return C2KV_OK;
}

static c2kv_status run_attention(const c2kv::Plan& p, void* ws, int src_kind, const char* name,
                                 const void* k, const void* v, const float* ks,
                                 const float* vs, const void* q, const void* k_suf,
                                 const void* v_suf, void* out, float* lse, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = timed(name, [&](hipEvent_t e0, hipEvent_t e1) {
    return c2kv::launch_attention(p, ws, src_kind, k, v, ks, vs, q, k_suf, v_suf, out, lse, s, e0,
                                  e1);
  });
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  if (!p.merges.empty() && !p.merge_in_kernel) {
    e = timed("merge", [&](hipEvent_t e0, hipEvent_t e1) {
      return c2kv::launch_merge(p, ws, out, lse, s, e0, e1);
    });
    if (e != hipSuccess) return hip_fail(e, "merge launch");
  }
  return C2KV_OK;
}

c2kv_status c2kv_attend(const c2kv_plan* plan, const void* k_pages, const void* v_pages,
                        const void* q, const void* k_suf, const void* v_suf, void* out,
                        float* lse, void* stream) {
  c2kv_status st;
  if (!check_plan(plan, &st)) return st;
  if (!check_io(q, k_suf, v_suf, out, &st)) return st;
  const c2kv::Plan& p = plan->p;
  if ((!k_pages || !v_pages) && p.n_pages > 0)
    return fail(C2KV_E_INVAL, "k_pages and v_pages must not be NULL");
  return run_attention(p, p.d_workspace, c2kv::kSrcPaged, "attn_paged", k_pages, v_pages,
                       nullptr, nullptr, q, k_suf, v_suf, out, lse, stream);
}

c2kv_status c2kv_compose_attend(const c2kv_plan* plan, const c2kv_pool* pool, const void* q,
                                const void* k_suf, const void* v_suf, void* out, float* lse,
                                void* stream) {
  c2kv_status st;
  if (!check_plan(plan, &st)) return st;
  const c2kv::Plan& p = plan->p;
  if (!check_pool(p, pool, &st)) return st;
  if (!check_io(q, k_suf, v_suf, out, &st)) return st;
  const int kind = pool->dtype == C2KV_I8 ? c2kv::kSrcPoolI8 : c2kv::kSrcPool;
  return run_attention(p, p.d_workspace, kind, "attn_pool", pool->k, pool->v, pool->k_scale,
                       pool->v_scale, q, k_suf, v_suf, out, lse, stream);
}

c2kv_status c2kv_compose_attend_static(const c2kv_plan* plan, const c2kv_pool* pool,
                                       const void* q, const void* k_suf, const void* v_suf,
                                       void* out, float* lse, void* stream) {
  if (!plan) return fail(C2KV_E_INVAL, "plan is NULL");
  const c2kv::Plan& p = plan->p;
  // checked before any HIP call: the tables and partials must fit the array
  if (p.ws.total > C2KV_STATIC_SCRATCH_BYTES)
    return fail(C2KV_E_WORKSPACE,
                "plan needs " + std::to_string(p.ws.total) + " bytes of scratch; the static "
                "array holds " + std::to_string(size_t(C2KV_STATIC_SCRATCH_BYTES)) +
                " (use c2kv_compose_attend with a workspace)");
  c2kv_status st;
  if (!check_pool(p, pool, &st)) return st;
  if (!check_io(q, k_suf, v_suf, out, &st)) return st;
  void* ws = nullptr;
  hipError_t e = c2kv::static_scratch(&ws);
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
  // this call's tables, over whatever the last call on this GPU left; the image
  // carries the zeroed merge counters as well
  e = hipMemcpyAsync(ws, p.image.data(), p.image.size(), hipMemcpyHostToDevice,
                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (tables into static scratch)");
  const int kind = pool->dtype == C2KV_I8 ? c2kv::kSrcPoolI8 : c2kv::kSrcPool;
  return run_attention(p, ws, kind, "attn_pool", pool->k, pool->v, pool->k_scale,
                       pool->v_scale, q, k_suf, v_suf, out, lse, stream);
}

c2kv_status c2kv_host_alloc(size_t bytes, void** host, void** device) {
  if (!host || !device || bytes == 0) return fail(C2KV_E_INVAL, "host_alloc: bad arguments");
  *host = nullptr;
  *device = nullptr;
  void* h = nullptr;
  hipError_t e = hipHostMalloc(&h, bytes, hipHostMallocMapped);
  if (e != hipSuccess) return hip_fail(e, "hipHostMalloc");
  void* d = nullptr;
  e = hipHostGetDevicePointer(&d, h, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(h);
    return hip_fail(e, "hipHostGetDevicePointer");
  }
  *host = h;
  *device = d;
  return C2KV_OK;
}

c2kv_status c2kv_host_free(void* host) {
  if (!host) return C2KV_OK;
  const hipError_t e = hipHostFree(host);
  return e == hipSuccess ? C2KV_OK : hip_fail(e, "hipHostFree");
}

c2kv_status c2kv_load(const c2kv_plan* plan, const c2kv_pool* src, const c2kv_pool* dst,
                      void* stream) {
  c2kv_status st;
  if (!check_plan(plan, &st)) return st;
  const c2kv::Plan& p = plan->p;
  if (!check_pool(p, src, &st) || !check_pool(p, dst, &st)) return st;
  if (src->dtype != dst->dtype) return fail(C2KV_E_INVAL, "load: pools of different dtypes");
  const size_t esz = src->dtype == C2KV_F32 ? 4 : src->dtype == C2KV_BF16 ? 2 : 1;
  const size_t row_bytes = esz * size_t(p.cfg.n_kv_heads) * size_t(p.cfg.head_dim);
  const size_t scale_bytes = sizeof(float) * size_t(p.cfg.n_kv_heads);
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto copy = [&](const void* from, void* to, size_t per_row, int64_t r0, int64_t r1) {
    return hipMemcpyAsync(static_cast<uint8_t*>(to) + size_t(r0) * per_row,
                          static_cast<const uint8_t*>(from) + size_t(r0) * per_row,
                          size_t(r1 - r0) * per_row, hipMemcpyDefault, s);
  };
  for (const auto& r : p.load_rows) {
    hipError_t e = copy(src->k, const_cast<void*>(dst->k), row_bytes, r.first, r.second);
    if (e == hipSuccess) e = copy(src->v, const_cast<void*>(dst->v), row_bytes, r.first, r.second);
    if (e == hipSuccess && src->dtype == C2KV_I8) {
      e = copy(src->k_scale, const_cast<float*>(dst->k_scale), scale_bytes, r.first, r.second);
      if (e == hipSuccess)
        e = copy(src->v_scale, const_cast<float*>(dst->v_scale), scale_bytes, r.first, r.second);
    }
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (load)");
  }
  return C2KV_OK;
}

c2kv_status c2kv_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.on = on != 0;
  return C2KV_OK;
}

c2kv_status c2kv_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto& kv : g_timing.recs)
    for (auto& r : kv.second) {
      g_timing.spare.push_back(r.a);
      g_timing.spare.push_back(r.b);
    }
  g_timing.recs.clear();
  return C2KV_OK;
}

c2kv_status c2kv_timing_read(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms || !launches) return fail(C2KV_E_INVAL, "NULL argument");
  std::lock_guard<std::mutex> lk(g_timing.mu);
  *total_ms = 0.0;
  *launches = 0;
  auto it = g_timing.recs.find(name);
  if (it == g_timing.recs.end()) return C2KV_OK;
  for (auto& r : it->second) {
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    *total_ms += ms;
    ++*launches;
  }
  return C2KV_OK;
}

}  // extern "C"
