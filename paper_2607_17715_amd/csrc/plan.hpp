// Host plan of the compose-and-attend path: everything that depends only on the
// composition descriptor and the attention shape, computed once per batch of
// requests and shared by every layer (the kept-token set of a segment is the
// same for all layers and heads).
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "c2kv.h"

namespace c2kv {

constexpr int kKeyTile = 64;        // keys per attention / compose tile
constexpr int kMaxSplits = 256;     // key splits of one row block (merge kernel's LDS table)
constexpr int kRowsPerWave = 32;    // query rows one wavefront owns (MFMA 32-wide)

// One attention workgroup: query rows [row0, row0 + nrows) of (request b,
// kv-head g) in t-major order (row r = t * G + head-within-group), over key
// tiles [tile0, tile1) of the combined tile list (cached tiles first, then the
// suffix tiles this row block can see).  partial < 0: write the final output;
// otherwise write partial `partial` of merge group `merge`.
struct WorkItem {
  int32_t b, g, row0, nrows, tile0, tile1, partial, merge;
  int32_t slot0, nslots;               // request b's composed slots [slot0, slot0 + nslots)
  int32_t page0;                       // request b's first page (its pages are consecutive)
  int32_t n_ranges;                    // 0: tiles [tile0, tile1); else item position
  int32_t rng[3];                      // i < tile1 runs through ranges [first, end) given
  int32_t pad;                         // as first | end << 16 (multi-range SIF items)
};

// Row block whose key splits are combined by the merge kernel.
struct MergeGroup {
  int32_t b, g, row0, nrows, part0, nsplit, pad0, pad1;
};

// Byte offsets of the device tables inside the workspace.
struct WorkspaceLayout {
  size_t req_slot0 = 0;   // int32 [B+1]
  size_t slot_info = 0;   // int32x2 [total_slots] (pool row, segment)
  size_t slot_pos = 0;    // int32 [total_slots]
  size_t seg_cs = 0;      // float2 [n_seg][D/2]   cos/sin(delta * theta_i)
  size_t suf_cs = 0;      // float2 [B][S][D/2]    cos/sin((span_end + t) * theta_i)
  size_t block_table = 0; // int32 [B][max_pages]
  size_t compose_tiles = 0; // int32x4 [n_compose_tiles] (first slot, keys, page, offset)
  size_t items = 0;       // WorkItem [n_items]
  size_t merges = 0;      // MergeGroup [n_merge]
  size_t counters = 0;    // int32 [n_merge], zero between launches
  size_t table_bytes = 0; // end of the tables (uploaded image size)
  size_t part_o = 0;      // activation dtype [n_partials][rows_per_block][D]
  size_t part_lse = 0;    // float [n_partials][rows_per_block]
  size_t total = 0;
};

struct Plan {
  c2kv_attn_cfg cfg{};
  int32_t batch = 0, suffix_len = 0, page_size = 64, n_segments = 0;
  int32_t group = 1;               // G = H_q / H_kv
  bool keys_pre_rope = false;      // pool keys stored before RoPE: per-slot cos/sin rows
  int32_t sif_n = 0, sif_block = 0, sif_sink = 0;   // SIF mask (sif_n > 0) instead of causal
  bool pool_compressed = false;    // slot k of a segment reads row seg_row0 + k
  std::vector<std::pair<int64_t, int64_t>> load_rows;   // merged [first, end) row ranges
  float qscale_log2 = 0.f;         // softmax scale * log2(e)
  float softmax_scale = 0.f;

  // layout (the bit-exact part)
  std::vector<int32_t> req_slot0;  // [B+1]
  std::vector<int32_t> span_end;   // [B]
  std::vector<int32_t> slot_src;   // [total]
  std::vector<int32_t> slot_seg;   // [total]
  std::vector<int32_t> slot_pos;   // [total] new position
  std::vector<int32_t> slot_delta; // [total]
  std::vector<int32_t> seg_delta;  // [n_seg]
  int64_t max_src_row = -1;

  // pages
  int32_t n_pages = 0, max_pages = 0;
  std::vector<int32_t> block_table;   // [B][max_pages]
  std::vector<int32_t> compose_tiles; // [n][4]

  // attention work decomposition
  int32_t rows_per_block = 128;
  std::vector<WorkItem> items;
  std::vector<MergeGroup> merges;
  int32_t n_partials = 0, max_splits = 1;
  bool merge_in_kernel = false;   // last split of a row block merges (else a merge kernel)

  // tables in float (host image)
  WorkspaceLayout ws;
  std::vector<uint8_t> image;       // [ws.table_bytes], uploaded verbatim

  // binding
  void* d_workspace = nullptr;
  size_t d_workspace_bytes = 0;
};

// Extraction-time attention with Structured Information Flow: a sequence of
// n_tokens original tokens followed by one C^2 token per block of `block` tokens.
struct SifShape { int32_t n_tokens, block, sink; };

// Builds the plan; returns C2KV_OK or an error with `err` set.  With `sif`, the
// request has no segments and its suffix is the SIF sequence.
c2kv_status build_plan(const c2kv_attn_cfg& cfg, const c2kv_compose_desc& desc,
                       int32_t suffix_len, const c2kv_plan_opts* opts, Plan& plan,
                       std::string& err, const SifShape* sif = nullptr);

// The SIF plan: batch sequences of n_tokens + ceil(n_tokens / block) tokens.
c2kv_status build_sif_plan(const c2kv_attn_cfg& cfg, int32_t batch, int32_t n_tokens,
                           int32_t block, int32_t sink, const c2kv_plan_opts* opts,
                           Plan& plan, std::string& err);

}  // namespace c2kv

struct c2kv_plan {
  c2kv::Plan p;
};
