// Host-only fuzz driver of the plan builder (plan.cpp), built with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer by test_plan_sanitize_cpu.py.
// It draws random descriptors, valid and invalid (negative rows, kept indices out
// of order or outside their span, positions near the int32 limit, bad page sizes
// and option values, SIF shapes), and checks every plan that is accepted: slot
// rows within the pool rows it reports, a block table that hands each request
// consecutive pages exactly once, compose tiles within their pages, work items
// whose rows and key tiles lie inside their request, and a workspace image that
// fits the reported size.  Usage: plan_fuzz <iterations> <seed>; prints
// "ok <accepted> rejected <n> sif_ok <n>" and returns 0, or names the first
// failed check and returns 1.
#include <cstdio>
#include <random>
#include <vector>
#include <set>
#include <algorithm>
#include "plan.hpp"
using namespace c2kv;
#define CHECK(c) do { if (!(c)) { std::printf("FAIL %s line %d iter %d\n", #c, __LINE__, it); return 1; } } while (0)
int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  std::mt19937_64 rng(argc > 2 ? atoll(argv[2]) : 12345);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int ok = 0, rej = 0, sif_ok = 0;
  for (int it = 0; it < iters; ++it) {
    c2kv_attn_cfg cfg{};
    const int hk[] = {1, 2, 4, 8};
    cfg.n_kv_heads = hk[U(0, 3)];
    cfg.n_q_heads = cfg.n_kv_heads * (1 << U(0, 4));
    cfg.head_dim = U(0, 9) == 0 ? 96 : (U(0, 1) ? 64 : 128);
    cfg.act_dtype = U(0, 3) == 0 ? C2KV_F32 : C2KV_BF16;
    cfg.rope_base = U(0, 20) == 0 ? -1.0 : 10000.0;
    cfg.softmax_scale = 0.f;
    c2kv_plan_opts o{};
    const int ps[] = {0, 64, 128, 256, 100};
    o.page_size = ps[U(0, 4)];
    const int rb[] = {0, 0, 64, 128, 256};
    o.rows_per_block = rb[U(0, 4)];
    o.kv_splits = U(0, 3) == 0 ? U(1, 9) : 0;
    o.merge_mode = U(0, 2);
    o.num_cus = U(0, 3) == 0 ? U(1, 300) : 0;
    Plan p; std::string err;
    if (U(0, 4) == 0) {  // SIF plan
      const int B = U(0, 3), n = U(0, 700), blk = U(0, 9), sink = U(-1, 20);
      c2kv_status st = build_sif_plan(cfg, B, n, blk, sink, &o, p, err);
      if (st == C2KV_OK) {
        ++sif_ok;
        CHECK(p.image.size() <= p.ws.total);
        for (const auto& w : p.items) CHECK(w.nrows > 0 && w.row0 >= 0);
      } else ++rej;
      continue;
    }
    const int B = U(0, 4) == 0 ? U(0, 1) : U(1, 5);
    std::vector<int32_t> req_off(std::max(B, 0) + 1, 0);
    std::vector<int64_t> row0; std::vector<int32_t> span, orig, newp, koff{0}, kept;
    const bool explicit_pos = U(0, 3) == 0;
    const bool compressed = U(0, 4) == 0;
    const int pool_rows = 4000;
    for (int b = 0; b < B; ++b) {
      const int ns = U(0, 4);
      for (int c = 0; c < ns; ++c) {
        const int sp = U(0, 6) == 0 ? 0 : U(1, 500);
        row0.push_back(U(0, 20) == 0 ? -U(1, 5) : U(0, pool_rows));
        span.push_back(U(0, 30) == 0 ? -1 : sp);
        orig.push_back(U(0, 10) == 0 ? U(0, 1 << 20) : 0);
        newp.push_back(U(0, 40) == 0 ? 0x7ffffff0 : U(0, 5000));
        std::vector<int> ks;
        for (int j = 0; j < sp; ++j) if (U(0, 99) < 30) ks.push_back(j);
        if (U(0, 30) == 0 && ks.size() > 1) std::swap(ks[0], ks[1]);
        if (U(0, 30) == 0) ks.push_back(sp);
        for (int j : ks) kept.push_back(j);
        koff.push_back(int32_t(kept.size()));
      }
      req_off[b + 1] = req_off[b] + ns;
    }
    if (U(0, 40) == 0 && B > 0) req_off[B] += 1;
    c2kv_compose_desc d{};
    d.batch = B;
    d.n_segments = int32_t(row0.size());
    d.req_seg_off = req_off.data();
    d.seg_row0 = row0.data(); d.seg_span = span.data(); d.seg_orig_pos0 = orig.data();
    d.seg_new_pos0 = explicit_pos ? newp.data() : nullptr;
    d.seg_kept_off = koff.data(); d.kept_idx = kept.data();
    d.key_encoding = U(0, 20) == 0 ? 5 : U(0, 1);
    d.pool_layout = compressed ? C2KV_POOL_COMPRESSED : C2KV_POOL_FULL;
    const int S = U(0, 30) == 0 ? 0 : (U(0, 1) ? U(1, 8) : U(1, 400));
    if (B == 0 && U(0, 1)) { d.req_seg_off = req_off.data(); }
    c2kv_status st = build_plan(cfg, d, S, &o, p, err);
    if (st != C2KV_OK) { ++rej; CHECK(!err.empty()); continue; }
    ++ok;
    // invariants
    CHECK(int(p.req_slot0.size()) == B + 1);
    const int64_t total = p.req_slot0[B];
    CHECK(int64_t(p.slot_src.size()) == total && int64_t(p.slot_pos.size()) == total);
    for (int64_t i = 0; i < total; ++i) CHECK(p.slot_src[i] >= 0 && p.slot_src[i] <= p.max_src_row);
    CHECK(int64_t(p.block_table.size()) == int64_t(B) * p.max_pages);
    std::set<int> used;
    for (int b = 0; b < B; ++b) {
      const int64_t n = p.req_slot0[b + 1] - p.req_slot0[b];
      const int64_t need = (n + p.page_size - 1) / p.page_size;
      for (int i = 0; i < p.max_pages; ++i) {
        const int v = p.block_table[size_t(b) * p.max_pages + i];
        if (i < need) { CHECK(v >= 0 && v < p.n_pages); CHECK(used.insert(v).second); }
        else CHECK(v == -1);
      }
    }
    CHECK(int(used.size()) == p.n_pages);
    CHECK(p.compose_tiles.size() % 4 == 0);
    for (size_t t = 0; t < p.compose_tiles.size(); t += 4) {
      CHECK(p.compose_tiles[t] >= 0 && p.compose_tiles[t] + p.compose_tiles[t + 1] <= total);
      CHECK(p.compose_tiles[t + 1] >= 1 && p.compose_tiles[t + 1] <= 64);
      CHECK(p.compose_tiles[t + 2] >= 0 && p.compose_tiles[t + 2] < p.n_pages);
      CHECK(p.compose_tiles[t + 3] >= 0 && p.compose_tiles[t + 3] + p.compose_tiles[t + 1] <= p.page_size);
    }
    CHECK(!p.items.empty());
    const int G = cfg.n_q_heads / cfg.n_kv_heads;
    for (const auto& w : p.items) {
      CHECK(w.b >= 0 && w.b < B && w.g >= 0 && w.g < cfg.n_kv_heads);
      CHECK(w.nrows >= 1 && w.nrows <= p.rows_per_block && w.row0 >= 0 && w.row0 + w.nrows <= G * S);
      CHECK(w.tile0 >= 0 && w.tile0 < w.tile1);
      const int64_t n = p.req_slot0[w.b + 1] - p.req_slot0[w.b];
      const int64_t tiles = (n + 63) / 64 + (S + 63) / 64;
      CHECK(w.tile1 <= tiles);
      CHECK(w.partial < p.n_partials && w.merge < int(p.merges.size()));
    }
    CHECK(p.image.size() <= p.ws.total && p.ws.total % 256 == 0);
  }
  std::printf("ok %d rejected %d sif_ok %d\n", ok, rej, sif_ok);
  return 0;
}
