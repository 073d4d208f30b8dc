// Work plan of one attention call (host only; see milo_plan.h): column tiles,
// gangs of workgroups, block parts and tail chunks dealt to the persistent
// workgroups of the attention kernel (Alg. 1 inference stage: the selected
// blocks plus each request's own KV).
#include "milo_plan.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

namespace milo {

// LDS of the attention kernel: a base region (projected query, weight tile and
// reductions, or the tail item's buffers) followed by kWaves rings of nslot
// fragments.
size_t attend_lds_base_bytes(int head_dim, int rk_pad_max, int rv_pad_max, bool half_w) {
  const size_t qsd = (size_t)rk_pad_max + 8;
  const size_t ws = half_w ? kTile / 2 + 8 : kWStride;
  const size_t loop = kCols * qsd * 2 + (size_t)kCols * ws * 2 + (size_t)kWaves * kCols * 4;
  // up-projection: the latent accumulator as bf16 [col][rank], or the segment
  // partials being combined (at most 4 slots x 3 rank tiles x 8 KiB), then the
  // per-wave column sums at the end of the region
  const size_t olat = (size_t)kCols * (rv_pad_max + 8) * 2;
  const size_t segs = (size_t)4 * 3 * 2 * 16 * 64 * 4;
  const size_t epi = (olat > segs ? olat : segs) + (size_t)kWaves * kCols * 4;
  const size_t tail = ((size_t)2 * kWaves * 32 + (size_t)kTailChunk * 32 + (size_t)kWaves * kMaxGroup * head_dim) * 4;
  size_t m = loop > epi ? loop : epi;
  m = m > tail ? m : tail;
  return (m + 1023) / 1024 * 1024;  // the fragment rings start here
}

size_t attend_ring_bytes(int nslot) { return (size_t)kWaves * nslot * kFragElems * 2; }

// ---------------------------------------------------------------------------
// Work schedule of one attention call.
//
// Query columns are numbered head-major (column g * N_g + i * G + h mod G of
// KV head g, request i, query head h; N_g = n_q * G) and cut into column tiles
// of at most kCols columns (make_tiling): whole KV heads per tile when a head
// has fewer than kCols columns, else either kCols-column pieces of each head or
// kCols consecutive columns that may span two heads, whichever needs clearly
// fewer tiles while still forming a wide gang.  Every column tile of a block re-reads
// the block's P factors, so fewer tiles means less P traffic and fewer padded
// MFMA columns.
//
// Work is cut into jobs: a block job is one part of a selected block (a range
// of whole 256-token tiles; large blocks are split so the work evens out) for a
// group of C column tiles, and a tail job is a bundle of up to C dense-tail
// chunks (one request, one KV head, kTailChunk tokens each).  A job's C items
// run on a "gang" of C workgroups of one XCD, so a block's P factors are fetched
// from HBM once and re-read by the gang's other workgroups from that XCD's L2.
// Workgroup b runs on XCD b % 8 (round-robin dispatch); the 32 workgroups of an
// XCD form 32 / C gangs, and the 32 mod C left over ("solo" workgroups) take
// single tail chunks.  Jobs are dealt to the gangs longest first (each to the
// gang with the least estimated work), then single jobs are moved or swapped
// between the most and the least loaded gang while that lowers the maximum; of
// several ways to split the blocks, the one with the smallest estimated
// makespan is kept.  Within a gang, tail jobs run first so their latency
// overlaps the start of the fragment streams.
//
// Tail chunks are planned up to a per-call capacity (the longest tail rounded
// up to a power of two of chunks, at most tail_cap), not to the exact tail
// lengths: the kernels read each request's length from their arguments and
// skip chunks past it, so a decode loop whose tails grow by one token per step
// reuses its plan until the longest tail doubles.
// ---------------------------------------------------------------------------
// Cost model (microseconds on an MI355X, least-squares fit to per-item kernel
// timings of the 7B-shaped layer, rms error 0.5 us): one fragment of the
// slowest wave's projection and up-projection streams, one fragment of its
// tile stream, the per-tile softmax and barriers, the per-item set-up, one
// round of the token-segment reduction, and one dense-tail chunk.
constexpr double kCostFragItem = 0.206, kCostFragTile = 0.153, kCostTile = 1.75, kCostItem = 2.43,
                 kCostSegRound = 0.61, kCostTail = 9.4;
constexpr int kPerXcd = kCUs / kXcds;  // workgroups per XCD

// Workgroups per gang for n_ct column tiles: a divisor of n_ct of at most one
// XCD's workgroups; the largest power of two (no solo workgroups), unless a
// divisor at least twice as large leaves at most two solos per XCD.
int gang_size(int n_ct) {
  int pow2 = 1;
  while (n_ct % (2 * pow2) == 0 && 2 * pow2 <= kPerXcd) pow2 *= 2;
  int best = 1;
  for (int c = 1; c <= std::min(n_ct, kPerXcd); ++c)
    if (n_ct % c == 0 && kPerXcd % c <= 2) best = c;
  return best >= 2 * pow2 ? best : pow2;
}

Tiling make_tiling(int n_kv, int N_g, bool head_tiles, int max_cols) {
  Tiling t;
  const int N = n_kv * N_g;
  if (head_tiles) {
    const int a = (N_g + kCols - 1) / kCols;
    t.geom = TileGeom{kTileHead, a, N_g, N};
    t.n_ct = n_kv * a;
  } else if (N_g < kCols) {
    const int a = std::max(1, std::min(kMaxTileHeads, max_cols / N_g));
    t.geom = TileGeom{kTilePacked, a, N_g, N};
    t.n_ct = (n_kv + a - 1) / a;
  } else {
    const int a = (N_g + kCols - 1) / kCols;
    const int n_head = n_kv * a, n_flat = (N + kCols - 1) / kCols;
    if (4 * n_flat <= 3 * n_head && 2 * gang_size(n_flat) >= n_flat) {
      t.geom = TileGeom{kTileFlat, 1, N_g, N};
      t.n_ct = n_flat;
    } else {
      t.geom = TileGeom{kTileHead, a, N_g, N};
      t.n_ct = n_head;
    }
  }
  for (int k = 0; k < t.n_ct; ++k) {
    int c0, cn;
    tile_range(t.geom, k, &c0, &cn);
    t.c0.push_back(c0);
    t.cn.push_back(cn);
    t.g0.push_back(c0 / N_g);
    t.nh.push_back((c0 + cn - 1) / N_g - c0 / N_g + 1);
  }
  return t;
}

// Latent rank tiles the busiest wave of a block accumulates (projection or value pass).
int max_owned(const BlockMeta& m) {
  const int nrt_k = m.rk_pad / 32, nrt_v = m.rv_pad / 32;
  const int ng = kWaves / v_segments(nrt_v);
  return std::max((nrt_k + kWaves - 1) / kWaves, (nrt_v + ng - 1) / ng);
}

bool build_schedule(const PlanInput& c, const int32_t* table, int n_sel, int n_q, int n_chunks, const Tiling& til,
                    int64_t program_cap, Schedule* out, std::string* err) {
  const int NK = c.d / 16;
  const bool any_recon = c.recon_region && std::any_of(table, table + n_sel, [&](int b) { return c.recon_region[b] >= 0; });
  if (any_recon && til.geom.mode != kTileHead) {
    *err = "reconstructed blocks need one KV head per column tile";
    return false;
  }
  auto is_dense = [&](int b) { return c.recon_region && c.recon_region[b] >= 0; };
  // the metadata the kernel sees for block b (for a reconstructed block: its
  // KV head 0; the other heads differ only in offsets)
  auto item_meta = [&](int b) { return is_dense(b) ? dense_meta(c.meta[b], c.recon_region[b], 0, c.d) : c.meta[b]; };
  auto item_cost = [&](const BlockMeta& m, int nt, int nh, bool dense) {
    const int nrt_k = m.rk_pad / 32, nks = m.rk_pad / 16, nrt_v = m.rv_pad / 32;
    const int nseg = v_segments(nrt_v), ng = kWaves / nseg;
    const int mk = (nrt_k + kWaves - 1) / kWaves, mv = (nrt_v + ng - 1) / ng;
    int rounds = 0;
    for (int h = nseg; h > 1; h /= 2) ++rounds;
    const double item_frags = dense ? 0.0 : nh * ((double)NK * mk + m.rv_pad / 32.0);
    const double tile_frags = nt * ((double)nks + 16.0 / nseg * mv);
    return kCostFragItem * item_frags + kCostFragTile * tile_frags + kCostTile * nt + kCostItem +
           kCostSegRound * rounds;
  };
  const int n_ct = til.n_ct;
  const int C = gang_size(n_ct);
  const int gangs_per_xcd = kPerXcd / C;
  const int n_gangs = kXcds * gangs_per_xcd, n_solo = kXcds * (kPerXcd % C);
  const int n_cg = n_ct / C;  // column-tile groups
  std::vector<int> grp_nh(n_cg, 1);  // most KV heads of a tile in the group
  for (int k = 0; k < n_ct; ++k) grp_nh[k / C] = std::max(grp_nh[k / C], til.nh[k]);
  out->gang = C;
  // a workgroup folds consecutive block items of one column tile into one
  // partial where the kernel keeps that partial in registers (at most two
  // latent rank tiles per wave)
  int max_own_all = 0;
  for (int j = 0; j < n_sel; ++j) max_own_all = std::max(max_own_all, max_owned(item_meta(table[j])));
  const bool fold = max_own_all <= 2;
  double total_blk = 0.0;
  for (int j = 0; j < n_sel; ++j) {
    const BlockMeta m = item_meta(table[j]);
    for (int cg = 0; cg < n_cg; ++cg) total_blk += item_cost(m, m.T_pad / kTile, grp_nh[cg], is_dense(table[j]));
  }
  // tail items, numbered (request, KV head, chunk); solo workgroups take the
  // first n_solo_items, the rest run in bundles of C on the gangs
  const int n_tail = n_q * c.n_kv * n_chunks;
  int n_solo_items = 0;
  if (n_solo > 0 && n_tail > 0) {
    const double per_gang = (total_blk + kCostTail * n_tail / C) / n_gangs;
    n_solo_items = (int)std::min<int64_t>(n_tail, (int64_t)n_solo * std::max(1, (int)(per_gang / kCostTail)));
  }
  auto tail_item = [&](int ti) {
    WorkItem w{};
    w.kind = kItemTail;
    w.req = ti / (c.n_kv * n_chunks);
    w.g = (ti / n_chunks) % c.n_kv;
    w.sub = ti % n_chunks;
    w.slot = w.sub;
    return w;
  };
  const double total = total_blk + kCostTail * (double)(n_tail - n_solo_items) / C;
  struct Part { int b, tile0, ntile; };
  struct Job { int part, cg, tail0, ntail; double cost; };  // part < 0: tail bundle
  // Jobs for one way of splitting the blocks: parts of at most `share` of a
  // gang's average work (and at most kMaxPartTiles tiles), longest first.
  auto make_jobs = [&](double share, std::vector<Part>& parts, std::vector<Job>& jobs) {
    const double target = std::max(1e-9, total / n_gangs * share);
    parts.clear();
    jobs.clear();
    for (int j = 0; j < n_sel; ++j) {
      const int b = table[j];
      const BlockMeta m = item_meta(b);
      const int nt = m.T_pad / kTile;
      const int np_cost =
          (int)std::min<double>(nt, std::max(1.0, std::ceil(item_cost(m, nt, 1, is_dense(b)) / target)));
      const int np = std::max(np_cost, (nt + kMaxPartTiles - 1) / kMaxPartTiles);
      for (int p = 0; p < np; ++p) {
        const int t_a = (int)((int64_t)nt * p / np), t_b = (int)((int64_t)nt * (p + 1) / np);
        parts.push_back({b, t_a, t_b - t_a});
      }
    }
    for (int p = 0; p < (int)parts.size(); ++p)
      for (int cg = 0; cg < n_cg; ++cg)
        jobs.push_back(
            {p, cg, 0, 0, item_cost(item_meta(parts[p].b), parts[p].ntile, grp_nh[cg], is_dense(parts[p].b))});
    for (int t0 = n_solo_items; t0 < n_tail; t0 += C) jobs.push_back({-1, 0, t0, std::min(C, n_tail - t0), kCostTail});
    std::stable_sort(jobs.begin(), jobs.end(), [](const Job& x, const Job& y) { return x.cost > y.cost; });
  };
  // Deal jobs (indices `idx`, longest first) to the gangs: each to the least
  // loaded gang, then improve by moving or swapping single jobs between the
  // most and the least loaded gang while that lowers the maximum.  Returns the
  // largest gang load.
  auto deal = [&](const std::vector<Job>& jobs, const std::vector<int>& idx,
                  std::vector<std::vector<int>>& lists) -> double {
    lists.assign(n_gangs, {});
    std::vector<double> load(n_gangs, 0.0);
    for (int k : idx) {
      const int best = (int)(std::min_element(load.begin(), load.end()) - load.begin());
      load[best] += jobs[k].cost;
      lists[best].push_back(k);
    }
    for (int iter = 0; iter < 4 * n_gangs; ++iter) {
      const int hi = (int)(std::max_element(load.begin(), load.end()) - load.begin());
      const int lo = (int)(std::min_element(load.begin(), load.end()) - load.begin());
      double best_max = load[hi];
      int bi = -1, bj = -1;  // job position in hi, and in lo (-1: move only)
      for (int i = 0; i < (int)lists[hi].size(); ++i) {
        const double ci = jobs[lists[hi][i]].cost;
        const double mv = std::max(load[hi] - ci, load[lo] + ci);
        if (mv < best_max - 1e-9) { best_max = mv; bi = i; bj = -1; }
        for (int j = 0; j < (int)lists[lo].size(); ++j) {
          const double cj = jobs[lists[lo][j]].cost;
          if (cj >= ci) continue;
          const double sw = std::max(load[hi] - ci + cj, load[lo] + ci - cj);
          if (sw < best_max - 1e-9) { best_max = sw; bi = i; bj = j; }
        }
      }
      if (bi < 0) break;
      const int ki = lists[hi][bi];
      lists[hi].erase(lists[hi].begin() + bi);
      load[hi] -= jobs[ki].cost;
      if (bj >= 0) {
        const int kj = lists[lo][bj];
        lists[lo].erase(lists[lo].begin() + bj);
        load[lo] -= jobs[kj].cost;
        lists[hi].push_back(kj);
        load[hi] += jobs[kj].cost;
      }
      lists[lo].push_back(ki);
      load[lo] += jobs[ki].cost;
    }
    // tail jobs first, then the longest block jobs.  Where items fold, the
    // block jobs go by column group first: consecutive items of one column
    // tile share one partial slot, so a gang writes (and the merge reads) one
    // partial per column group instead of one per block.  Where they do not,
    // the order stays by length alone, which keeps the column groups of one
    // block close in time on different gangs (its P is read while cached).
    for (auto& l : lists)
      std::stable_sort(l.begin(), l.end(), [&](int x, int y) {
        if ((jobs[x].part < 0) != (jobs[y].part < 0)) return jobs[x].part < 0;
        if (fold && jobs[x].cg != jobs[y].cg) return jobs[x].cg < jobs[y].cg;
        return jobs[x].cost > jobs[y].cost;
      });
    return *std::max_element(load.begin(), load.end());
  };
  // the split whose dealt schedule has the smallest estimated makespan
  std::vector<Part> parts;
  std::vector<Job> jobs;
  {
    double best = 1e300, best_share = 1.0;
    for (double share : {1.5, 1.0, 0.8, 0.67, 0.5, 0.33}) {
      make_jobs(share, parts, jobs);
      std::vector<int> idx(jobs.size());
      std::iota(idx.begin(), idx.end(), 0);
      std::vector<std::vector<int>> lists;
      const double mk = deal(jobs, idx, lists);
      if (mk < best - 1e-9) { best = mk; best_share = share; }
    }
    make_jobs(best_share, parts, jobs);
  }
  const int n_parts = (int)parts.size();
  out->n_parts = n_parts;
  for (const Part& pt : parts) {
    const BlockMeta m = item_meta(pt.b);
    out->rk_pad_max = std::max(out->rk_pad_max, m.rk_pad);
    out->rv_pad_max = std::max(out->rv_pad_max, m.rv_pad);
    out->max_own = std::max(out->max_own, max_owned(m));
  }

  // LDS plan: the projected query, weight tile and a 6-slot fragment ring,
  // the rest for the program (fewer launches would cost the ring); when even a
  // short program leaves no room for that (ranks above 512), the weight tile
  // in two 128-token halves and a 4-slot ring; failing that, no ring
  // run buffers sized for this plan's items: the most KV heads of a tile and
  // the most tiles of a part
  int max_nh = 1, max_pt = 1;
  for (int k = 0; k < n_ct; ++k) max_nh = std::max(max_nh, til.nh[k]);
  for (const Part& pt : parts) max_pt = std::max(max_pt, pt.ntile);
  out->run_cap = run_cap_for(max_nh, max_pt, c.p_int8);
  const size_t run_bytes = (size_t)kWaves * kRunBufs * out->run_cap * sizeof(int2);
  const size_t short_prog = 16 * sizeof(WorkItem) + run_bytes;
  auto room_for = [&](bool half_w) {
    const size_t b = attend_lds_base_bytes(c.d, out->rk_pad_max, out->rv_pad_max, half_w);
    return b < (size_t)kLdsBytes ? kLdsBytes - b : 0;
  };
  size_t cap;
  if (room_for(false) >= attend_ring_bytes(6) + short_prog) {
    out->half_w = false;
    cap = room_for(false) - attend_ring_bytes(6);
  } else if (room_for(true) >= attend_ring_bytes(4) + short_prog) {
    out->half_w = true;
    cap = room_for(true) - attend_ring_bytes(4);
  } else {
    out->half_w = false;
    cap = room_for(false);
  }
  if (program_cap >= 0) cap = std::min(cap, (size_t)program_cap);
  for (int L = 1; L <= (1 << 20); L *= 2) {
    std::vector<std::vector<unsigned char>> progs((size_t)L * kCUs);
    std::vector<WgProgram> entries((size_t)L * kCUs);
    std::vector<int32_t> slot_count((size_t)n_ct, 0);
    size_t max_prog = 0;
    // the items of one workgroup's program: slot groups, then its bytes
    auto emit = [&](int l, int wg, std::vector<WorkItem>& items) {
      // consecutive block items of one column tile share a slot (when the
      // kernel folds them); slots of a tile are numbered densely
      int first = -1, last = -1;
      for (int i = 0; i < (int)items.size(); ++i) {
        WorkItem& w = items[i];
        if (w.kind != kItemBlock) continue;
        const bool cont = fold && first >= 0 && items[first].sub == w.sub;
        if (cont) {
          w.slot = items[first].slot;
        } else {
          if (last >= 0) items[last].flags |= kItemFlush;
          first = i;
          w.flags |= kItemFirst;
          w.slot = slot_count[(size_t)w.sub]++;
        }
        last = i;
      }
      if (last >= 0) items[last].flags |= kItemFlush;
      WgProgram& e = entries[(size_t)l * kCUs + wg];
      e = WgProgram{};
      if (items.empty()) return;
      std::vector<unsigned char>& pb = progs[(size_t)l * kCUs + wg];
      pb.resize(items.size() * sizeof(WorkItem));
      std::memcpy(pb.data(), items.data(), pb.size());
      e.n_items = (int32_t)items.size();
      e.words = (int32_t)(pb.size() / 4);
      // LDS: the items, then every wave's run buffers
      max_prog = std::max(max_prog, pb.size() + run_bytes);
    };
    for (int l = 0; l < L; ++l) {
      std::vector<int> idx;
      for (size_t k = l; k < jobs.size(); k += L) idx.push_back((int)k);
      std::vector<std::vector<int>> lists;
      deal(jobs, idx, lists);
      for (int gang = 0; gang < n_gangs; ++gang) {
        for (int j = 0; j < C; ++j) {
          const int wg = (gang % kXcds) + kXcds * ((gang / kXcds) * C + j);
          std::vector<WorkItem> items;
          for (int k : lists[gang]) {
            const Job& jb = jobs[k];
            if (jb.part < 0) {
              if (j < jb.ntail) items.push_back(tail_item(jb.tail0 + j));
              continue;
            }
            const int tile = jb.cg * C + j;
            const Part& pt = parts[jb.part];
            WorkItem w{};
            const bool dense = is_dense(pt.b);
            w.blk = dense ? dense_meta(c.meta[pt.b], c.recon_region[pt.b], til.g0[tile], c.d) : c.meta[pt.b];
            w.kind = kItemBlock;
            w.g = til.g0[tile];
            w.sub = tile;
            w.req = til.c0[tile];
            w.tile0 = pt.tile0;
            w.ntile = pt.ntile;
            w.flags = (lg_rank_groups(w.blk.rv_pad / 32) << kItemLgNgShift) | ((til.cn[tile] - 1) << kItemColsShift) |
                      ((til.nh[tile] - 1) << kItemHeadsShift) | (c.p_int8 ? kItemInt8 : 0) |
                      (dense ? kItemDense : 0) | (pt.b == c.causal_block ? kItemCausal : 0);
            items.push_back(w);
          }
          emit(l, wg, items);
        }
      }
      // solo workgroups: solo s takes tail items s, s + n_solo, ... of the
      // solo share, spread over the launches
      for (int s = 0; s < n_solo; ++s) {
        const int wg = (s % kXcds) + kXcds * (C * gangs_per_xcd + s / kXcds);
        std::vector<WorkItem> items;
        for (int q = s, r = 0; q < n_solo_items; q += n_solo, ++r)
          if (r % L == l) items.push_back(tail_item(q));
        emit(l, wg, items);
      }
    }
    const size_t prog_bytes = (max_prog + 255) / 256 * 256;
    if (prog_bytes > cap) continue;
    // assemble: the entry table, every program at a 16-byte aligned offset,
    // then the slot counts
    size_t off = entries.size() * sizeof(WgProgram);
    for (size_t k = 0; k < progs.size(); ++k) {
      entries[k].off = (int64_t)off;
      off += progs[k].size();
    }
    out->count_off = (int64_t)((off + 15) / 16 * 16);
    off = (size_t)out->count_off + slot_count.size() * sizeof(int32_t);
    out->bytes.assign(std::max<size_t>(off, 16), 0);
    std::memcpy(out->bytes.data(), entries.data(), entries.size() * sizeof(WgProgram));
    for (size_t k = 0; k < progs.size(); ++k)
      if (!progs[k].empty()) std::memcpy(out->bytes.data() + entries[k].off, progs[k].data(), progs[k].size());
    std::memcpy(out->bytes.data() + out->count_off, slot_count.data(), slot_count.size() * sizeof(int32_t));
    out->n_block_slots = 0;
    for (int32_t k : slot_count) out->n_block_slots = std::max(out->n_block_slots, (int)k);
    out->n_launch = L;
    out->prog_bytes = (int)prog_bytes;
    return true;
  }
  *err = "work schedule does not fit in LDS";
  return false;
}

void build_recon_plan(const BlockMeta* meta, const int32_t* table, int n_sel, const char* recon, int n_kv, int d,
                      std::vector<int64_t>* region, ReconPlan* out, const int32_t* rope_pos) {
  out->blocks.clear();
  out->tasks.clear();
  out->elems = 0;
  const int D = n_kv * d;
  std::vector<std::vector<int2>> queue(kXcds);
  std::vector<double> load(kXcds, 0.0);
  for (int j = 0; j < n_sel; ++j) {
    const int b = table[j];
    if (!recon[j]) continue;
    const BlockMeta& m = meta[b];
    ReconBlock rb{};
    rb.src = m;
    rb.dst = out->elems;
    rb.pos0 = rope_pos ? rope_pos[b] : -1;
    (*region)[b] = out->elems;
    out->elems += 2 * (int64_t)m.T_pad * D;
    const int i = (int)out->blocks.size();
    out->blocks.push_back(rb);
    // K, then V: each side's tasks (heads x tiles) on the least loaded XCD
    for (int side = 0; side < 2; ++side) {
      const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
      const int r_pad = side ? m.rv_pad : m.rk_pad;
      for (int t = 0; t < m.T_pad / kTile; ++t)
        for (int g = 0; g < n_kv; ++g) queue[x].push_back(make_int2(i, (t << 8) | (g << 1) | side));
      load[x] += (double)(m.T_pad / kTile) * n_kv * (r_pad / 32 + 2);  // rank steps + epilogue
    }
  }
  size_t longest = 0;
  for (const auto& q : queue) longest = std::max(longest, q.size());
  out->tasks.assign(longest * kXcds, make_int2(-1, 0));
  for (int x = 0; x < kXcds; ++x)
    for (size_t k = 0; k < queue[x].size(); ++k) out->tasks[k * kXcds + x] = queue[x][k];
}

}  // namespace milo
