// Host plan builder: validation, the kept-token slot table with span-preserving
// positions (Section 3.2 "Output and Reuse"), per-segment and per-suffix-token
// RoPE cos/sin tables computed in float64, the page assignment and the
// attention work list.  Pure host code: no HIP call happens here, so plans can
// be built and inspected on a machine without a GPU.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <sstream>

#include "plan.hpp"

namespace c2kv {
namespace {

constexpr int64_t kI32Max = std::numeric_limits<int32_t>::max();

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int32_t ceil_div(int64_t a, int64_t b) { return static_cast<int32_t>((a + b - 1) / b); }

template <typename... Args>
std::string fmt(Args&&... args) {
  std::ostringstream os;
  (os << ... << args);
  return os.str();
}

// theta_i = base^(-2i/D), i < D/2, in float64 (RoPE frequencies).
std::vector<double> rope_theta(int D, double base) {
  std::vector<double> th(D / 2);
  for (int i = 0; i < D / 2; ++i) th[i] = std::pow(base, -2.0 * i / D);
  return th;
}

}  // namespace

c2kv_status build_plan(const c2kv_attn_cfg& cfg, const c2kv_compose_desc& d,
                       int32_t suffix_len, const c2kv_plan_opts* opts, Plan& p,
                       std::string& err, const SifShape* sif) {
  // ---- attention shape ----------------------------------------------------
  if (cfg.n_q_heads < 1 || cfg.n_kv_heads < 1 || cfg.n_q_heads % cfg.n_kv_heads != 0) {
    err = fmt("n_q_heads (", cfg.n_q_heads, ") must be a positive multiple of n_kv_heads (",
              cfg.n_kv_heads, ")");
    return C2KV_E_INVAL;
  }
  if (cfg.head_dim <= 0 || cfg.head_dim % 2 != 0) {
    err = fmt("head_dim must be positive and even, got ", cfg.head_dim);
    return C2KV_E_INVAL;
  }
  if (cfg.head_dim != 64 && cfg.head_dim != 128) {
    err = fmt("head_dim ", cfg.head_dim, " not built (64 or 128)");
    return C2KV_E_UNSUPPORTED;
  }
  if (cfg.act_dtype != C2KV_F32 && cfg.act_dtype != C2KV_BF16) {
    err = "act_dtype must be C2KV_F32 or C2KV_BF16";
    return C2KV_E_INVAL;
  }
  if (!(cfg.rope_base > 0.0) || !std::isfinite(cfg.rope_base)) {
    err = "rope_base must be positive and finite";
    return C2KV_E_INVAL;
  }
  if (!std::isfinite(cfg.softmax_scale)) {
    err = "softmax_scale must be finite";
    return C2KV_E_INVAL;
  }
  if (suffix_len < 1) {
    err = fmt("suffix_len must be >= 1, got ", suffix_len);
    return C2KV_E_INVAL;
  }

  // ---- options --------------------------------------------------------------
  c2kv_plan_opts o{};
  if (opts) o = *opts;
  if (o.page_size == 0) o.page_size = 64;
  if (o.page_size < 0 || o.page_size % kKeyTile != 0) {
    err = fmt("page_size must be a positive multiple of ", kKeyTile, ", got ", o.page_size);
    return C2KV_E_INVAL;
  }
  if (o.rows_per_block != 0 && o.rows_per_block != 64 && o.rows_per_block != 128 &&
      o.rows_per_block != 256) {
    err = fmt("rows_per_block must be 0, 64, 128 or 256, got ", o.rows_per_block);
    return C2KV_E_INVAL;
  }
  if (o.kv_splits < 0 || o.num_cus < 0) {
    err = "kv_splits and num_cus must be >= 0";
    return C2KV_E_INVAL;
  }
  if (o.merge_mode < 0 || o.merge_mode > 2) {
    err = fmt("merge_mode must be 0, 1 or 2, got ", o.merge_mode);
    return C2KV_E_INVAL;
  }
  if (o.num_cus == 0) o.num_cus = 256;

  // ---- descriptor -----------------------------------------------------------
  const int32_t B = d.batch;
  if (B < 1) { err = fmt("batch must be >= 1, got ", B); return C2KV_E_INVAL; }
  if (d.n_segments < 0) { err = "n_segments must be >= 0"; return C2KV_E_INVAL; }
  if (!d.req_seg_off) { err = "req_seg_off is NULL"; return C2KV_E_INVAL; }
  if (d.req_seg_off[0] != 0 || d.req_seg_off[B] != d.n_segments) {
    err = "req_seg_off must start at 0 and end at n_segments";
    return C2KV_E_INVAL;
  }
  for (int b = 0; b < B; ++b)
    if (d.req_seg_off[b + 1] < d.req_seg_off[b]) {
      err = fmt("req_seg_off decreases at request ", b);
      return C2KV_E_INVAL;
    }
  const int32_t nseg = d.n_segments;
  if (nseg > 0 && (!d.seg_row0 || !d.seg_span || !d.seg_orig_pos0 || !d.seg_kept_off)) {
    err = "segment arrays must not be NULL";
    return C2KV_E_INVAL;
  }
  if (nseg > 0 && d.seg_kept_off[0] != 0) { err = "seg_kept_off[0] must be 0"; return C2KV_E_INVAL; }
  for (int c = 0; c < nseg; ++c) {
    if (d.seg_kept_off[c + 1] < d.seg_kept_off[c]) {
      err = fmt("seg_kept_off decreases at segment ", c);
      return C2KV_E_INVAL;
    }
  }
  const int64_t total_kept = nseg > 0 ? d.seg_kept_off[nseg] : 0;
  if (total_kept > 0 && !d.kept_idx) { err = "kept_idx is NULL"; return C2KV_E_INVAL; }
  if (total_kept > kI32Max) { err = "too many kept tokens"; return C2KV_E_UNSUPPORTED; }

  p = Plan{};
  p.cfg = cfg;
  p.batch = B;
  p.suffix_len = suffix_len;
  p.page_size = o.page_size;
  p.n_segments = nseg;
  p.group = cfg.n_q_heads / cfg.n_kv_heads;
  if (d.key_encoding != C2KV_KEYS_ROPE_AT_ORIG && d.key_encoding != C2KV_KEYS_PRE_ROPE) {
    err = "key_encoding must be C2KV_KEYS_ROPE_AT_ORIG or C2KV_KEYS_PRE_ROPE";
    return C2KV_E_INVAL;
  }
  p.keys_pre_rope = d.key_encoding == C2KV_KEYS_PRE_ROPE;
  if (d.pool_layout != C2KV_POOL_FULL && d.pool_layout != C2KV_POOL_COMPRESSED) {
    err = "pool_layout must be C2KV_POOL_FULL or C2KV_POOL_COMPRESSED";
    return C2KV_E_INVAL;
  }
  p.pool_compressed = d.pool_layout == C2KV_POOL_COMPRESSED;
  p.softmax_scale = cfg.softmax_scale > 0.f ? cfg.softmax_scale
                                            : static_cast<float>(1.0 / std::sqrt(double(cfg.head_dim)));
  p.qscale_log2 = static_cast<float>(double(p.softmax_scale) * 1.4426950408889634);

  // ---- slot table: segments in request order, kept indices ascending --------
  p.req_slot0.assign(B + 1, 0);
  p.span_end.assign(B, 0);
  p.seg_delta.assign(nseg, 0);
  p.slot_src.reserve(total_kept);
  p.slot_seg.reserve(total_kept);
  p.slot_pos.reserve(total_kept);
  p.slot_delta.reserve(total_kept);
  for (int b = 0; b < B; ++b) {
    int64_t cursor = 0, end = 0;
    for (int c = d.req_seg_off[b]; c < d.req_seg_off[b + 1]; ++c) {
      const int64_t span = d.seg_span[c];
      const int64_t row0 = d.seg_row0[c];
      const int64_t orig0 = d.seg_orig_pos0[c];
      const int64_t new0 = d.seg_new_pos0 ? int64_t(d.seg_new_pos0[c]) : cursor;
      if (span < 1) { err = fmt("seg_span[", c, "] must be >= 1, got ", span); return C2KV_E_INVAL; }
      if (row0 < 0) { err = fmt("seg_row0[", c, "] < 0"); return C2KV_E_INVAL; }
      if (orig0 < 0 || new0 < 0) { err = fmt("negative position at segment ", c); return C2KV_E_INVAL; }
      const int64_t delta = new0 - orig0;
      if (new0 + span > kI32Max || orig0 + span > kI32Max || delta > kI32Max || delta < -kI32Max) {
        err = fmt("positions of segment ", c, " overflow int32");
        return C2KV_E_INVAL;
      }
      p.seg_delta[c] = static_cast<int32_t>(delta);
      int64_t prev = -1;
      int64_t first_row = -1, last_row = -1;
      for (int k = d.seg_kept_off[c]; k < d.seg_kept_off[c + 1]; ++k) {
        const int64_t j = d.kept_idx[k];
        if (j < 0 || j >= span) {
          err = fmt("kept index ", j, " of segment ", c, " outside [0, ", span, ")");
          return C2KV_E_INVAL;
        }
        if (j <= prev) {
          err = fmt("kept indices of segment ", c, " are not strictly ascending");
          return C2KV_E_INVAL;
        }
        prev = j;
        const int64_t src = row0 + (p.pool_compressed ? int64_t(k - d.seg_kept_off[c]) : j);
        if (first_row < 0) first_row = src;
        last_row = src;
        if (src > kI32Max) { err = "pool row beyond int32 range"; return C2KV_E_UNSUPPORTED; }
        p.slot_src.push_back(static_cast<int32_t>(src));
        p.slot_seg.push_back(c);
        p.slot_pos.push_back(static_cast<int32_t>(new0 + j));
        p.slot_delta.push_back(static_cast<int32_t>(delta));
        p.max_src_row = std::max<int64_t>(p.max_src_row, src);
      }
      if (first_row >= 0) p.load_rows.push_back({first_row, last_row + 1});
      cursor = new0 + span;               // span-preserving: advance by n, not m
      // the query tokens start past every placed span (explicit placements may
      // put the furthest span before the last segment)
      end = std::max(end, new0 + span);
    }
    if (end + suffix_len - 1 > kI32Max) {
      err = fmt("suffix positions of request ", b, " overflow int32");
      return C2KV_E_INVAL;
    }
    p.span_end[b] = static_cast<int32_t>(end);
    p.req_slot0[b + 1] = static_cast<int32_t>(p.slot_src.size());
  }

  // rows the load step copies: segment ranges sorted and merged
  std::sort(p.load_rows.begin(), p.load_rows.end());
  {
    std::vector<std::pair<int64_t, int64_t>> merged;
    for (const auto& r : p.load_rows) {
      if (!merged.empty() && r.first <= merged.back().second)
        merged.back().second = std::max(merged.back().second, r.second);
      else
        merged.push_back(r);
    }
    p.load_rows.swap(merged);
  }

  // ---- pages: each request gets ceil(N_b / page) consecutive pages ----------
  const int PS = p.page_size;
  int64_t pages = 0;
  int32_t maxp = 1;
  for (int b = 0; b < B; ++b) {
    const int64_t n = p.req_slot0[b + 1] - p.req_slot0[b];
    maxp = std::max(maxp, ceil_div(n, PS));
  }
  p.max_pages = maxp;
  p.block_table.assign(size_t(B) * maxp, -1);
  for (int b = 0; b < B; ++b) {
    const int64_t n = p.req_slot0[b + 1] - p.req_slot0[b];
    const int32_t np = ceil_div(n, PS);
    for (int i = 0; i < np; ++i) p.block_table[size_t(b) * maxp + i] = static_cast<int32_t>(pages + i);
    pages += np;
  }
  if (pages > kI32Max) { err = "too many pages"; return C2KV_E_UNSUPPORTED; }
  // the kernels find a tile's page by multiplying with a 32-bit reciprocal of the
  // tiles per page, exact while tiles * tiles-per-page stays below 2^32
  {
    int64_t max_tiles = 0;
    for (int b = 0; b < B; ++b)
      max_tiles = std::max<int64_t>(max_tiles, ceil_div(p.req_slot0[b + 1] - p.req_slot0[b],
                                                        kKeyTile));
    if ((max_tiles + 4) * (PS / kKeyTile) >= (int64_t(1) << 32)) {
      err = fmt("page_size ", PS, " too large for requests of ", max_tiles, " key tiles");
      return C2KV_E_UNSUPPORTED;
    }
  }
  p.n_pages = static_cast<int32_t>(pages);
  // compose tiles carry what their workgroup needs, so that it starts with one
  // scalar load: first slot, keys in the tile, page and offset in the page
  for (int b = 0; b < B; ++b) {
    const int64_t n = p.req_slot0[b + 1] - p.req_slot0[b];
    for (int t = 0; t < ceil_div(n, kKeyTile); ++t) {
      const int64_t k0 = int64_t(t) * kKeyTile;
      p.compose_tiles.push_back(static_cast<int32_t>(p.req_slot0[b] + k0));
      p.compose_tiles.push_back(static_cast<int32_t>(std::min<int64_t>(kKeyTile, n - k0)));
      p.compose_tiles.push_back(p.block_table[size_t(b) * maxp + k0 / PS]);
      p.compose_tiles.push_back(static_cast<int32_t>(k0 % PS));
    }
  }

  // ---- attention work list ---------------------------------------------------
  const int64_t G = p.group, S = suffix_len;
  const int64_t R = G * S;            // query rows per (request, kv-head)
  int RB = o.rows_per_block;
  // fp32 products (32x32x2 MFMA: eight times the instructions of bf16 per
  // product) favour twice the workgroups of 64-row blocks below 256 rows
  if (RB == 0) RB = R >= 256 ? 256 : R > 64 && cfg.act_dtype == C2KV_BF16 ? 128 : 64;
  p.rows_per_block = RB;
  // 8 wavefronts at 2 per SIMD fill a CU; 64-row blocks have 4 and run two to a CU
  const int wgs_per_cu = RB == 64 ? 2 : 1;
  const int64_t target = int64_t(o.num_cus) * wgs_per_cu;
  const int32_t n_rb = ceil_div(R, RB);
  // A group is one row block of one (request, kv-head) and the key tiles it reads
  // (composed tiles first, then suffix tiles), as a list of [first, end) ranges.
  struct Group {
    int32_t b, g, row0, nrows, tiles;
    std::vector<std::pair<int32_t, int32_t>> ranges;
  };
  std::vector<Group> groups;
  int64_t total_tiles = 0;
  for (int b = 0; b < B; ++b) {
    const int64_t n = p.req_slot0[b + 1] - p.req_slot0[b];
    const int32_t nct = ceil_div(n, kKeyTile);
    for (int g = 0; g < cfg.n_kv_heads; ++g)
      for (int rb = 0; rb < n_rb; ++rb) {
        const int32_t row0 = rb * RB;
        const int32_t nrows = static_cast<int32_t>(std::min<int64_t>(RB, R - row0));
        const int64_t tmin = row0 / G, tmax = (row0 + nrows - 1) / G;   // suffix tokens
        Group gr{b, g, row0, nrows, 0, {}};
        if (sif && tmin >= sif->n_tokens) {
          // C^2 rows only: the sink, the blocks of these C^2 tokens, and the C^2
          // tokens up to the last of them (keys are suffix tiles: nct = 0)
          const int64_t j0 = tmin - sif->n_tokens, j1 = tmax - sif->n_tokens;
          std::vector<std::pair<int32_t, int32_t>> r;
          if (sif->sink > 0) r.push_back({0, ceil_div(sif->sink, kKeyTile)});
          r.push_back({static_cast<int32_t>(j0 * sif->block / kKeyTile),
                       ceil_div(std::min<int64_t>((j1 + 1) * sif->block, sif->n_tokens), kKeyTile)});
          r.push_back({static_cast<int32_t>(sif->n_tokens / kKeyTile),
                       ceil_div(sif->n_tokens + j1 + 1, kKeyTile)});
          std::sort(r.begin(), r.end());
          for (const auto& x : r) {
            if (!gr.ranges.empty() && x.first <= gr.ranges.back().second)
              gr.ranges.back().second = std::max(gr.ranges.back().second, x.second);
            else
              gr.ranges.push_back(x);
          }
        } else {
          gr.ranges.push_back({0, nct + ceil_div(tmax + 1, kKeyTile)});
        }
        for (const auto& x : gr.ranges) gr.tiles += x.second - x.first;
        total_tiles += gr.tiles;
        groups.push_back(std::move(gr));
      }
  }
  // Key splits only add parallelism where the row blocks alone leave CUs idle;
  // with at least one row block per CU they would only add partials, a merge
  // and a second round of workgroups.
  const bool split = int64_t(groups.size()) < target;
  const int64_t per_item =
      split ? std::max<int64_t>(1, (total_tiles + target - 1) / target) : INT32_MAX;
  std::vector<WorkItem> items;
  for (const Group& gr : groups) {
    // a SIF row block over several key ranges is one item that runs through
    // them in turn (no partials, no merge), when its tiles fit 16-bit fields
    if (sif && gr.ranges.size() > 1 && gr.ranges.size() <= 3 &&
        gr.ranges.back().second < 65536 && o.kv_splits == 0) {
      WorkItem w{gr.b, gr.g, gr.row0, gr.nrows, 0, gr.tiles, -1, -1,
                 p.req_slot0[gr.b], p.req_slot0[gr.b + 1] - p.req_slot0[gr.b],
                 p.block_table[size_t(gr.b) * p.max_pages], int32_t(gr.ranges.size()),
                 {0, 0, 0}, 0};
      for (size_t ri = 0; ri < gr.ranges.size(); ++ri)
        w.rng[ri] = gr.ranges[ri].first | (gr.ranges[ri].second << 16);
      items.push_back(w);
      continue;
    }
    // splits of each range, at most kMaxSplits in all
    std::vector<int32_t> nsr;
    int32_t ns = 0;
    for (const auto& x : gr.ranges) {
      const int32_t len = x.second - x.first;
      int32_t k = o.kv_splits > 0 ? o.kv_splits : ceil_div(len, per_item);
      // With splits, take as many as one round of workgroups holds: the longest
      // item keeps its tile count and the CUs the rounding left idle get work.
      // Measured: int8 layer (one workgroup per CU) -1.2 %; at two workgroups
      // per CU (decode) -7 % where the items then hold at most 4 tiles, and up
      // to +5 % for the long uncompressed contexts, which keep the rounded count.
      if (o.kv_splits == 0 && split) {
        const int32_t fill = static_cast<int32_t>(
            std::min<int64_t>(len, target / int64_t(groups.size()) / int64_t(gr.ranges.size())));
        if (fill > k && (wgs_per_cu == 1 || ceil_div(len, fill) <= 4)) k = fill;
      }
      k = std::max(1, std::min({k, len, kMaxSplits / int32_t(gr.ranges.size())}));
      nsr.push_back(k);
      ns += k;
    }
    p.max_splits = std::max(p.max_splits, ns);
    int32_t part0 = -1, merge = -1;
    if (ns > 1) {
      part0 = p.n_partials;
      merge = static_cast<int32_t>(p.merges.size());
      p.merges.push_back({gr.b, gr.g, gr.row0, gr.nrows, part0, ns, 0, 0});
      p.n_partials += ns;
    }
    int32_t k = 0;
    for (size_t ri = 0; ri < gr.ranges.size(); ++ri) {
      const int32_t first = gr.ranges[ri].first, len = gr.ranges[ri].second - first;
      for (int s = 0; s < nsr[ri]; ++s, ++k) {
        const int32_t t0 = first + static_cast<int32_t>(int64_t(len) * s / nsr[ri]);
        const int32_t t1 = first + static_cast<int32_t>(int64_t(len) * (s + 1) / nsr[ri]);
        items.push_back({gr.b, gr.g, gr.row0, gr.nrows, t0, t1, ns > 1 ? part0 + k : -1, merge,
                         p.req_slot0[gr.b], p.req_slot0[gr.b + 1] - p.req_slot0[gr.b],
                         p.block_table[size_t(gr.b) * p.max_pages], 0, {0, 0, 0}, 0});
      }
    }
  }
  // never chosen automatically: each split's agent-scope release writes back its
  // XCD's whole L2 and the last split's acquire invalidates it, which costs the
  // other workgroups there their cached keys and values (measured 2-5x slower
  // than the separate merge kernel)
  p.merge_in_kernel = o.merge_mode == 1;

  // XCD-aware order.  Workgroups are dealt to the 8 XCDs round-robin by index,
  // and each XCD has its own L2.  Items of one (request, kv-head) read the same
  // keys, values and queries, so they are kept on one XCD: (b, g) pairs go to the
  // least-loaded XCD queue, queues hold their heaviest items first, and the
  // grid interleaves the queues.
  constexpr int kXcds = 8;
  std::vector<std::vector<WorkItem>> queue(kXcds);
  std::vector<int64_t> load(kXcds, 0);
  {
    std::vector<std::pair<int64_t, int64_t>> pairs;   // (-tiles, b * H + g)
    std::vector<int64_t> tiles_of(size_t(B) * cfg.n_kv_heads, 0);
    for (const WorkItem& w : items) tiles_of[size_t(w.b) * cfg.n_kv_heads + w.g] += w.tile1 - w.tile0;
    for (size_t k = 0; k < tiles_of.size(); ++k) pairs.push_back({-tiles_of[k], int64_t(k)});
    std::sort(pairs.begin(), pairs.end());
    std::vector<int> bin_of(tiles_of.size(), 0);
    for (const auto& pr : pairs) {
      const int x = static_cast<int>(std::min_element(load.begin(), load.end()) - load.begin());
      bin_of[pr.second] = x;
      load[x] += -pr.first;
    }
    for (const WorkItem& w : items) queue[bin_of[size_t(w.b) * cfg.n_kv_heads + w.g]].push_back(w);
    for (auto& q : queue)
      std::stable_sort(q.begin(), q.end(), [](const WorkItem& a, const WorkItem& b) {
        return (a.tile1 - a.tile0) > (b.tile1 - b.tile0);
      });
  }
  std::vector<size_t> head(kXcds, 0);
  for (size_t n = 0; n < items.size(); ++n) {
    int x = static_cast<int>(n % kXcds);
    if (head[x] >= queue[x].size()) {           // this queue ran dry: take the fullest one
      size_t best = 0;
      for (int y = 0; y < kXcds; ++y)
        if (queue[y].size() - head[y] > best) { best = queue[y].size() - head[y]; x = y; }
    }
    p.items.push_back(queue[x][head[x]++]);
  }

  // ---- workspace image --------------------------------------------------------
  const int D = cfg.head_dim, H = D / 2;
  const int64_t total = static_cast<int64_t>(p.slot_src.size());
  WorkspaceLayout& w = p.ws;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t at = off; off = align256(off + std::max<size_t>(bytes, 4)); return at; };
  w.req_slot0 = take(sizeof(int32_t) * (B + 1));
  w.slot_info = take(sizeof(int32_t) * 2 * total);
  w.slot_pos = take(sizeof(int32_t) * total);
  // one cos/sin row per segment (angle delta * theta_i), or per slot for keys
  // stored before RoPE (angle p_new * theta_i); slot_info's second field is the row
  const int64_t cs_rows = p.keys_pre_rope ? total : nseg;
  w.seg_cs = take(sizeof(float) * 2 * size_t(std::max<int64_t>(cs_rows, 1)) * H);
  w.suf_cs = take(sizeof(float) * 2 * size_t(B) * S * H);
  w.block_table = take(sizeof(int32_t) * p.block_table.size());
  w.compose_tiles = take(sizeof(int32_t) * p.compose_tiles.size());
  w.items = take(sizeof(WorkItem) * p.items.size());
  w.merges = take(sizeof(MergeGroup) * p.merges.size());
  w.counters = take(sizeof(int32_t) * p.merges.size());
  w.table_bytes = off;
  const size_t act_bytes = cfg.act_dtype == C2KV_F32 ? 4 : 2;
  w.part_o = take(act_bytes * size_t(p.n_partials) * RB * D);
  w.part_lse = take(sizeof(float) * size_t(p.n_partials) * RB);
  w.total = off;

  p.image.assign(w.table_bytes, 0);
  auto put = [&](size_t at, const void* src, size_t bytes) {
    if (bytes) std::memcpy(p.image.data() + at, src, bytes);
  };
  put(w.req_slot0, p.req_slot0.data(), sizeof(int32_t) * (B + 1));
  {
    int32_t* si = reinterpret_cast<int32_t*>(p.image.data() + w.slot_info);
    for (int64_t i = 0; i < total; ++i) {
      si[2 * i] = p.slot_src[i];
      si[2 * i + 1] = p.keys_pre_rope ? static_cast<int32_t>(i) : p.slot_seg[i];
    }
  }
  put(w.slot_pos, p.slot_pos.data(), sizeof(int32_t) * total);
  put(w.block_table, p.block_table.data(), sizeof(int32_t) * p.block_table.size());
  put(w.compose_tiles, p.compose_tiles.data(), sizeof(int32_t) * p.compose_tiles.size());
  put(w.items, p.items.data(), sizeof(WorkItem) * p.items.size());
  put(w.merges, p.merges.data(), sizeof(MergeGroup) * p.merges.size());

  // cos/sin tables: angles in float64, rounded once to float32
  const std::vector<double> theta = rope_theta(D, cfg.rope_base);
  float* seg_cs = reinterpret_cast<float*>(p.image.data() + w.seg_cs);
  for (int64_t c = 0; c < cs_rows; ++c) {
    const double turn = p.keys_pre_rope ? double(p.slot_pos[c]) : double(p.seg_delta[c]);
    for (int i = 0; i < H; ++i) {
      const double ang = turn * theta[i];
      seg_cs[(size_t(c) * H + i) * 2 + 0] = static_cast<float>(std::cos(ang));
      seg_cs[(size_t(c) * H + i) * 2 + 1] = static_cast<float>(std::sin(ang));
    }
  }
  // suffix token t sits at span_end + t; with SIF, original token t at t and C^2
  // token j at the position of the last token of its block
  if (sif) {
    p.sif_n = sif->n_tokens;
    p.sif_block = sif->block;
    p.sif_sink = sif->sink;
  }
  auto suffix_pos = [&](int b, int64_t t) -> int64_t {
    if (!sif) return p.span_end[b] + t;
    if (t < sif->n_tokens) return t;
    return std::min<int64_t>((t - sif->n_tokens + 1) * sif->block, sif->n_tokens) - 1;
  };
  float* suf_cs = reinterpret_cast<float*>(p.image.data() + w.suf_cs);
  for (int b = 0; b < B; ++b)
    for (int64_t t = 0; t < S; ++t)
      for (int i = 0; i < H; ++i) {
        const double ang = double(suffix_pos(b, t)) * theta[i];
        const size_t k = ((size_t(b) * S + t) * H + i) * 2;
        suf_cs[k + 0] = static_cast<float>(std::cos(ang));
        suf_cs[k + 1] = static_cast<float>(std::sin(ang));
      }
  return C2KV_OK;
}

c2kv_status build_sif_plan(const c2kv_attn_cfg& cfg, int32_t batch, int32_t n_tokens,
                           int32_t block, int32_t sink, const c2kv_plan_opts* opts, Plan& p,
                           std::string& err) {
  if (batch < 1 || n_tokens < 1 || block < 1 || sink < 0 || sink > n_tokens) {
    err = fmt("SIF shape: need batch >= 1, n_tokens >= 1, block >= 1, 0 <= sink <= n_tokens; got ",
              batch, ", ", n_tokens, ", ", block, ", ", sink);
    return C2KV_E_INVAL;
  }
  const int64_t m = (int64_t(n_tokens) + block - 1) / block;
  if (n_tokens + m > kI32Max / 2) { err = "SIF sequence too long"; return C2KV_E_UNSUPPORTED; }
  // no composed segments: the whole [original | C^2] sequence is the suffix
  std::vector<int32_t> seg_off(size_t(batch) + 1, 0);
  const int32_t kept_off0 = 0;
  c2kv_compose_desc d{};
  d.batch = batch;
  d.n_segments = 0;
  d.req_seg_off = seg_off.data();
  d.seg_kept_off = &kept_off0;
  const SifShape sif{n_tokens, block, sink};
  return build_plan(cfg, d, static_cast<int32_t>(n_tokens + m), opts, p, err, &sif);
}

}  // namespace c2kv
