// Host-only check of the attention work plan (milo_plan.cpp): for every case
// read from stdin, build the plan and decode its programs, then check that
//  - the column tiles partition the head-major query columns and tile_of()
//    agrees with tile_range() for every column;
//  - every 256-token tile of every selected block is covered exactly once per
//    column tile, and every planned tail chunk (request, KV head, chunk)
//    exactly once;
//  - block items carry their tile's first column, KV heads and column count,
//    their block's rank-group split, at most kMaxPartTiles tiles, and derive
//    fewer fragment runs per wave than the plan's run buffers hold;
//  - partial slots: consecutive block items of one workgroup and column tile
//    form a group (first item flagged first, last flagged flush) that owns one
//    slot; slots of a tile are numbered densely from 0 and the plan's slot count
//    of every tile says how many (folding only where the kernel folds);
//  - every program fits the LDS region the plan reserves for it.
//  - reconstructed blocks (recon 1: every selected block, 2: every other one):
//    their items are dense items naming the tile's KV head in the block's
//    region, per-head column tiles; the reconstruction tasks cover every
//    (block, K or V, KV head, 256-token tile) exactly once, each block side's
//    tasks on one XCD, and the regions lie back to back.
// Case format (whitespace separated):
//   n_kv d G n_q n_chunks program_cap int8 recon gemv n_blocks  (T rk rv) x n_blocks  n_sel  table...
// (gemv: the projection runs as a GEMV, so tiles that pack heads hold at most
// kGemvCols columns)
#include <cstdio>
#include <cstring>
#include <map>
#include <set>
#include <string>
#include <tuple>
#include <algorithm>
#include <vector>

#include "milo_plan.h"

using namespace milo;

static int fails = 0;
#define CHECK(cond, ...)                         \
  do {                                           \
    if (!(cond)) {                               \
      std::printf("case %d: ", case_no);         \
      std::printf(__VA_ARGS__);                  \
      std::printf("\n");                         \
      ++fails;                                   \
      return;                                    \
    }                                            \
  } while (0)

static void run_case(int case_no, int n_kv, int d, int G, int n_q, int n_chunks, long long program_cap, int i8,
                     int recon_mode, int gemv, const std::vector<int>& T, const std::vector<int>& rk, const std::vector<int>& rv,
                     const std::vector<int>& table) {
  const int nb = (int)T.size();
  std::vector<BlockMeta> meta(nb);
  int64_t off = 0;
  for (int b = 0; b < nb; ++b) {
    BlockMeta& m = meta[b];
    m.T = T[b];
    m.T_pad = (T[b] + kTile - 1) / kTile * kTile;
    m.rk_pad = (rk[b] + 31) / 32 * 32;
    m.rv_pad = (rv[b] + 31) / 32 * 32;
    const int D = n_kv * d;
    m.off_pk = off;
    off += (int64_t)m.T_pad * m.rk_pad;
    m.off_rk = off;
    off += (int64_t)m.rk_pad * D;
    m.off_pv = off;
    off += (int64_t)m.T_pad * m.rv_pad;
    m.off_rv = off;
    off += (int64_t)m.rv_pad * D;
  }
  const int N_g = n_q * G, N = n_kv * N_g;
  // reconstructed blocks
  std::vector<char> recon(table.size(), 0);
  for (size_t j = 0; j < table.size(); ++j) recon[j] = recon_mode == 1 || (recon_mode == 2 && j % 2 == 0);
  const bool any_recon = std::any_of(recon.begin(), recon.end(), [](char x) { return x != 0; });
  std::vector<int64_t> region(nb, -1);
  ReconPlan rp;
  if (any_recon) build_recon_plan(meta.data(), table.data(), (int)table.size(), recon.data(), n_kv, d, &region, &rp);
  {
    const int D = n_kv * d;
    int64_t next = 0;
    std::map<std::tuple<int, int, int, int>, int> task_seen;
    std::map<std::pair<int, int>, int> xcd_of;  // (recon block, side) -> XCD
    int i = 0;
    for (size_t j = 0; j < table.size(); ++j) {
      const int b = table[j];
      if (!recon[j]) {
        CHECK(region[b] == -1, "latent block %d has a region", b);
        continue;
      }
      CHECK(region[b] == next && rp.blocks[i].dst == next, "block %d region %lld, expected %lld", b,
            (long long)region[b], (long long)next);
      CHECK(std::memcmp(&rp.blocks[i].src, &meta[b], sizeof(BlockMeta)) == 0, "reconstruction block %d metadata", i);
      next += 2LL * meta[b].T_pad * D;
      ++i;
    }
    CHECK(i == (int)rp.blocks.size() && rp.elems == next, "reconstruction blocks / buffer size");
    CHECK(rp.tasks.size() % kXcds == 0, "task count not a multiple of the XCDs");
    for (size_t k = 0; k < rp.tasks.size(); ++k) {
      const int2 tk = rp.tasks[k];
      if (tk.x < 0) continue;
      CHECK(tk.x < (int)rp.blocks.size(), "task %zu block %d", k, tk.x);
      const int side = tk.y & 1, g = (tk.y >> 1) & 127, t = tk.y >> 8;
      CHECK(g < n_kv && t < rp.blocks[tk.x].src.T_pad / kTile, "task %zu out of range", k);
      const int seen_now = ++task_seen[std::make_tuple(tk.x, side, g, t)];
      CHECK(seen_now == 1, "task %zu repeated", k);
      auto it = xcd_of.find({tk.x, side});
      if (it == xcd_of.end()) xcd_of[{tk.x, side}] = (int)(k % kXcds);
      else CHECK(it->second == (int)(k % kXcds), "block %d side %d spread over XCDs", tk.x, side);
    }
    size_t want = 0;
    for (const ReconBlock& r : rp.blocks) want += 2 * (size_t)n_kv * (r.src.T_pad / kTile);
    CHECK(task_seen.size() == want, "%zu tasks, want %zu", task_seen.size(), want);
  }
  const Tiling til = make_tiling(n_kv, N_g, any_recon, gemv ? kGemvCols : kCols);
  if (any_recon) CHECK(til.geom.mode == kTileHead, "reconstructed blocks without per-head tiles");
  if (gemv && N_g <= kGemvCols)
    for (int k = 0; k < til.n_ct; ++k) CHECK(til.cn[k] <= kGemvCols, "GEMV tile %d has %d columns", k, til.cn[k]);
  // tiles partition the columns; tile_of agrees with tile_range
  {
    int next = 0;
    for (int k = 0; k < til.n_ct; ++k) {
      CHECK(til.c0[k] == next, "tile %d starts at %d, expected %d", k, til.c0[k], next);
      CHECK(til.cn[k] >= 1 && til.cn[k] <= kCols, "tile %d has %d columns", k, til.cn[k]);
      CHECK(til.nh[k] >= 1 && til.nh[k] <= kMaxTileHeads, "tile %d spans %d heads", k, til.nh[k]);
      for (int cc = til.c0[k]; cc < til.c0[k] + til.cn[k]; ++cc)
        CHECK(tile_of(til.geom, cc) == k, "column %d: tile_of %d, in tile %d", cc, tile_of(til.geom, cc), k);
      next += til.cn[k];
    }
    CHECK(next == N, "tiles cover %d of %d columns", next, N);
  }
  Schedule sch;
  std::string err;
  PlanInput pin{meta.data(), n_kv, d, i8 != 0};
  pin.recon_region = any_recon ? region.data() : nullptr;
  if (!build_schedule(pin, table.data(), (int)table.size(), n_q, n_chunks, til, program_cap, &sch, &err)) {
    CHECK(false, "plan failed: %s", err.c_str());
  }
  const bool fold = sch.max_own <= 2;
  const auto* entries = reinterpret_cast<const WgProgram*>(sch.bytes.data());
  const int32_t* slot_count = reinterpret_cast<const int32_t*>(sch.bytes.data() + sch.count_off);
  CHECK(sch.count_off + (int64_t)til.n_ct * 4 <= (int64_t)sch.bytes.size(), "slot counts outside the plan");
  // coverage counters
  std::map<std::pair<int, int>, std::vector<int>> cover;  // (block, column tile) -> per token tile count
  for (int b : table)
    for (int k = 0; k < til.n_ct; ++k) cover[{b, k}].assign(meta[b].T_pad / kTile, 0);
  std::vector<int> tail_seen((size_t)n_q * n_kv * n_chunks, 0);
  std::vector<std::set<int>> slots_of_tile(til.n_ct);
  const size_t run_bytes = (size_t)kWaves * kRunBufs * sch.run_cap * sizeof(int2);
  CHECK(sch.run_cap >= 1 && sch.run_cap <= kRunCap, "run buffer of %d entries", sch.run_cap);
  for (int e = 0; e < sch.n_launch * kCUs; ++e) {
    const WgProgram& p = entries[e];
    if (p.n_items == 0) continue;
    CHECK(p.off % 16 == 0 && p.off + (int64_t)p.words * 4 <= sch.count_off, "program %d outside the plan", e);
    CHECK((size_t)p.words * 4 == (size_t)p.n_items * sizeof(WorkItem), "program %d size", e);
    CHECK((size_t)p.words * 4 + run_bytes <= (size_t)sch.prog_bytes, "program %d exceeds its LDS region", e);
    std::vector<WorkItem> items(p.n_items);
    std::memcpy(items.data(), sch.bytes.data() + p.off, (size_t)p.n_items * sizeof(WorkItem));
    int group_tile = -1, group_slot = -1;
    bool open = false;
    for (int i = 0; i < p.n_items; ++i) {
      const WorkItem& w = items[i];
      if (w.kind == kItemTail) {
        CHECK(w.req >= 0 && w.req < n_q && w.g >= 0 && w.g < n_kv && w.sub >= 0 && w.sub < n_chunks,
              "tail item out of range");
        CHECK(w.slot == w.sub, "tail item slot");
        tail_seen[((size_t)w.req * n_kv + w.g) * n_chunks + w.sub]++;
        continue;
      }
      CHECK(w.kind == kItemBlock, "unknown item kind %d", w.kind);
      const int k = w.sub;
      CHECK(k >= 0 && k < til.n_ct, "block item tile %d", k);
      CHECK(w.req == til.c0[k] && w.g == til.g0[k], "block item tile fields");
      CHECK(((w.flags >> kItemColsShift) & 63) + 1 == til.cn[k], "block item column count");
      CHECK(((w.flags >> kItemHeadsShift) & 7) + 1 == til.nh[k], "block item head count");
      const bool dense = (w.flags & kItemDense) != 0;
      int b = -1;
      if (dense) {
        for (int x = 0; x < nb; ++x)
          if (region[x] >= 0 && w.blk.off_pk >= region[x] && w.blk.off_pk < region[x] + 2LL * meta[x].T_pad * n_kv * d)
            b = x;
        CHECK(b >= 0, "dense item outside every region");
        const BlockMeta want = dense_meta(meta[b], region[b], til.g0[k], d);
        CHECK(std::memcmp(&want, &w.blk, sizeof(BlockMeta)) == 0 && til.nh[k] == 1, "dense item metadata");
      } else {
        for (int x = 0; x < nb; ++x)
          if (meta[x].off_pk == w.blk.off_pk) b = x;
        CHECK(b >= 0 && std::memcmp(&meta[b], &w.blk, sizeof(BlockMeta)) == 0, "block item metadata");
        CHECK(region[b] < 0, "block %d is reconstructed but has a latent item", b);
      }
      CHECK(((w.flags >> kItemLgNgShift) & 3) == lg_rank_groups(w.blk.rv_pad / 32), "rank groups field");
      CHECK(((w.flags & kItemInt8) != 0) == (i8 != 0), "INT8 flag");
      CHECK(w.ntile >= 1 && w.ntile <= kMaxPartTiles && w.tile0 >= 0 && w.tile0 + w.ntile <= meta[b].T_pad / kTile,
            "block item tile range");
      CHECK(!dense || !i8, "dense item in an INT8 plan");
      auto it = cover.find({b, k});
      CHECK(it != cover.end(), "block %d is not selected", b);
      for (int t = w.tile0; t < w.tile0 + w.ntile; ++t) it->second[t]++;
      // the runs of every wave, derived as the kernel does with a distance to
      // the reconstruction buffer: a dense item's fragments lie in its head's
      // region (shifted by that distance), any other item's in its own block's
      // factors (bf16 fragments; INT8 runs count 512-byte units)
      const int kDelta = 1 << 24;
      int64_t lo, hi;  // element range of the item's fragments
      if (dense) {
        lo = w.blk.off_pk + (int64_t)kDelta * kFragElems;
        hi = lo + 2LL * w.blk.T_pad * d;
      } else {
        lo = std::min({meta[b].off_pk, meta[b].off_rk, meta[b].off_pv, meta[b].off_rv});
        hi = meta[b].off_rv + (int64_t)meta[b].rv_pad * n_kv * d;
      }
      for (int wave = 0; wave < kWaves; ++wave) {
        int runs = 0;
        bool outside = false;
        block_runs(w.blk, w.g, til.nh[k], w.tile0, w.ntile, wave, d, lg_rank_groups(w.blk.rv_pad / 32),
                   (w.flags & kItemInt8) != 0, [&](int x, int n) {
                     ++runs;
                     const int kind = (n >> kRunKindShift) & 3, cnt = n & kRunCountMask;
                     if (kind == kRunScale) return;  // scale units: checked by the layout tests
                     const int64_t unit = kind == kRunI8 ? kFragElems / 2 : kFragElems;  // elements per unit index
                     if ((int64_t)x * unit < lo || ((int64_t)x + cnt) * unit > hi) outside = true;
                   }, dense, kDelta);
        CHECK(runs <= sch.run_cap - 1, "%d runs exceed the plan's run buffer of %d", runs, sch.run_cap);
        CHECK(!outside, "%s item: wave %d reads outside its block", dense ? "dense" : "latent", wave);
      }
      // slot groups
      const bool first = (w.flags & kItemFirst) != 0, flush = (w.flags & kItemFlush) != 0;
      if (first) {
        CHECK(!open, "group opened twice");
        CHECK(slots_of_tile[k].insert(w.slot).second, "slot %d of tile %d used by two groups", w.slot, k);
        group_tile = k;
        group_slot = w.slot;
        open = true;
      } else {
        CHECK(open && fold && group_tile == k && group_slot == w.slot, "item continues no group");
      }
      if (flush) open = false;
      CHECK(fold || (first && flush), "items fold where the kernel does not");
      // a group never spans items of another kind or tile
      if (!flush) CHECK(i + 1 < p.n_items && items[i + 1].kind == kItemBlock && items[i + 1].sub == k, "group break");
    }
    CHECK(!open, "group left open");
  }
  for (auto& kv : cover)
    for (size_t t = 0; t < kv.second.size(); ++t)
      CHECK(kv.second[t] == 1, "block %d tile %zu column tile %d covered %d times", kv.first.first, t,
            kv.first.second, kv.second[t]);
  for (size_t x = 0; x < tail_seen.size(); ++x) CHECK(tail_seen[x] == 1, "tail item %zu seen %d times", x, tail_seen[x]);
  int max_slots = 0;
  for (int k = 0; k < til.n_ct; ++k) {
    const int n = (int)slots_of_tile[k].size();
    CHECK(slot_count[k] == n, "tile %d: slot count %d, groups %d", k, slot_count[k], n);
    if (n) CHECK(*slots_of_tile[k].rbegin() == n - 1, "tile %d: slots not dense", k);
    max_slots = std::max(max_slots, n);
  }
  CHECK(sch.n_block_slots == max_slots, "n_block_slots %d, busiest tile %d", sch.n_block_slots, max_slots);
  const size_t base = attend_lds_base_bytes(d, sch.rk_pad_max, sch.rv_pad_max, sch.half_w);
  CHECK(base + (size_t)sch.prog_bytes + (sch.half_w ? attend_ring_bytes(4) : 0) <= (size_t)kLdsBytes,
        "LDS over budget");
  std::printf("case %d: tiles %d (mode %d) gang %d launches %d parts %d slots %d prog %d B\n", case_no, til.n_ct,
              til.geom.mode, sch.gang, sch.n_launch, sch.n_parts, sch.n_block_slots, sch.prog_bytes);
}

int main() {
  int case_no = 0;
  int n_kv, d, G, n_q, n_chunks, nb, i8, rc, gv;
  long long cap;
  while (std::scanf("%d %d %d %d %d %lld %d %d %d %d", &n_kv, &d, &G, &n_q, &n_chunks, &cap, &i8, &rc, &gv, &nb) ==
         10) {
    std::vector<int> T(nb), rk(nb), rv(nb);
    for (int b = 0; b < nb; ++b)
      if (std::scanf("%d %d %d", &T[b], &rk[b], &rv[b]) != 3) return 2;
    int n_sel;
    if (std::scanf("%d", &n_sel) != 1) return 2;
    std::vector<int> table(n_sel);
    for (int j = 0; j < n_sel; ++j)
      if (std::scanf("%d", &table[j]) != 1) return 2;
    run_case(case_no++, n_kv, d, G, n_q, n_chunks, cap, i8, rc, gv, T, rk, rv, table);
  }
  std::printf("%s (%d cases)\n", fails ? "FAIL" : "OK", case_no);
  return fails ? 1 : 0;
}
