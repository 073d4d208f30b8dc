// Host side of the C ABI in include/milo.h: argument validation, the packed
// cache (Sec. 4.2 factors stored per block with per-block ranks, Sec. 4.3),
// the per-call work plan and the kernel launches of one decode step
// (Alg. 1 inference stage: attention over the selected blocks plus the
// request's own KV).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <vector>

#include "milo.h"
#include "milo_internal.h"

using namespace milo;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  const int code = (e == hipErrorOutOfMemory) ? MILO_ERR_OUT_OF_MEMORY : MILO_ERR_HIP;
  return fail(code, "%s: %s", what, hipGetErrorString(e));
}

#define MILO_HIP(call)                                    \
  do {                                                    \
    hipError_t e_ = (call);                               \
    if (e_ != hipSuccess) return hip_fail(e_, #call);     \
  } while (0)

constexpr int64_t kAlignElems = kFragElems;  // every packed factor starts on a whole fragment

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

int64_t env_byte_cap() {
  const char* s = std::getenv("MILO_MAX_DEVICE_BYTES");
  if (!s || !*s) return -1;
  return std::strtoll(s, nullptr, 10);
}

// LDS bytes a workgroup program may use at most, from MILO_MAX_PROGRAM_BYTES
// (unset: no cap beyond what LDS leaves).  A small cap splits a step's work
// over several attention launches; it exists so that path can be exercised.
int64_t env_program_cap() {
  const char* s = std::getenv("MILO_MAX_PROGRAM_BYTES");
  if (!s || !*s) return -1;
  return std::strtoll(s, nullptr, 10);
}

// Timing hooks (measurement only).
struct TimingState {
  std::mutex mu;
  bool enabled = false;
  std::vector<hipEvent_t> pool;
  std::vector<hipEvent_t> recorded;  // groups of 4: attend kernel start / end, merge kernel start / end
};
TimingState g_timing;

}  // namespace

struct milo_cache {
  int device = -1;
  int n_blocks = 0, n_kv = 0, d = 0;
  std::vector<int32_t> T, rk, rv;
  std::vector<BlockMeta> meta;
  uint16_t* data = nullptr;
  int64_t data_elems = 0;
  // per-call workspace
  float* part_o = nullptr;
  float2* part_ml = nullptr;
  int64_t part_cols_slots = 0;  // capacity in (column, slot) pairs
  unsigned char* plan_d = nullptr;       // program table + programs of the attention launches
  unsigned char* plan_pinned = nullptr;  // staging copy for the upload
  int64_t plan_cap = 0;
  int32_t* tail_len_d = nullptr;
  int64_t tail_len_cap = 0;
  int32_t* tail_len_pinned = nullptr;
  // the plan of the previous call
  std::vector<int32_t> plan_key;
  int n_launch = 0, n_slots = 0, n_block_slots = 0, max_rt = 0, nslot = 0, rk_pad_max = 0, n_ct = 0;
  int64_t count_off = 0;  // byte offset of the plan's slot counts
  int prog_bytes = 0, ring_offset = 0;
  size_t lds = 0;
};

namespace {

FactorGeom geom_of(const milo_cache& c, int b, int which) {
  FactorGeom f{};
  f.kind = which;
  f.n_kv = c.n_kv;
  f.d = c.d;
  const int D = c.n_kv * c.d;
  f.T_pad = (int)round_up(c.T[b], kTile);
  switch (which) {
    case kPK: f.rows = c.T[b]; f.cols = c.rk[b]; f.r_pad = (int)round_up(c.rk[b], 32); break;
    case kRK: f.rows = c.rk[b]; f.cols = D; f.r_pad = (int)round_up(c.rk[b], 32); break;
    case kPV: f.rows = c.T[b]; f.cols = c.rv[b]; f.r_pad = (int)round_up(c.rv[b], 32); break;
    default:  f.rows = c.rv[b]; f.cols = D; f.r_pad = (int)round_up(c.rv[b], 32); break;
  }
  return f;
}

int64_t factor_offset(const BlockMeta& m, int which) {
  switch (which) {
    case kPK: return m.off_pk;
    case kRK: return m.off_rk;
    case kPV: return m.off_pv;
    default:  return m.off_rv;
  }
}

// ---------------------------------------------------------------------------
// Work schedule of one attention call.
//
// Work is cut into jobs: a block job is one part of a selected block (a range
// of whole 256-token tiles; large blocks are split so the work evens out) for
// a group of C 64-column tiles of query columns, and a tail job is C 256-token
// chunks of one request's dense KV.  Each job covers S_kv KV heads x C at once:
// its S = S_kv * C work items run on a "gang" of S workgroups of one XCD
// (S_kv = KV heads rounded up to a power of two; C = the largest power of two
// dividing the number of column tiles with S <= 32), so a block's P factors are
// fetched from HBM once and re-read by the other heads and column tiles from
// that XCD's L2.  Workgroup j of a gang takes head j % S_kv and column tile
// (or tail chunk) j / S_kv of the job's group.  Jobs are dealt to
// the gangs longest first (each to the gang with the least estimated work),
// then single jobs are moved or swapped between the most and the least loaded
// gang while that lowers the maximum; of several ways to split the blocks, the
// one with the smallest estimated makespan is kept.  Within a gang, tail jobs
// run first so their latency overlaps the start of the fragment streams.  Workgroup b runs on XCD b % 8 (round-robin dispatch), so
// gang k on XCD k % 8 uses workgroups (k % 8) + 8 * ((k / 8) * S + j), j < S.
// ---------------------------------------------------------------------------
// Cost model (microseconds on an MI355X, least-squares fit to per-item kernel
// timings of the 7B-shaped layer, rms error 0.5 us): one fragment of the
// slowest wave's projection and up-projection streams, one fragment of its
// tile stream, the per-tile softmax and barriers, the per-item set-up, one
// round of the token-segment reduction, and one dense-tail chunk.
constexpr double kCostFragItem = 0.206, kCostFragTile = 0.153, kCostTile = 1.75, kCostItem = 2.43,
                 kCostSegRound = 0.61, kCostTail = 9.4;

struct Schedule {
  std::vector<unsigned char> bytes;  // WgProgram[n_launch * kCUs], then the programs
  int n_launch = 0, n_parts = 0, prog_bytes = 0, rk_pad_max = 32, rv_pad_max = 32, max_own = 1;
  int n_block_slots = 0;  // block-group slots of the busiest (KV head, column tile)
  bool half_w = false;    // the weight tile in 128-token halves (LDS is short)
  int64_t count_off = 0;  // byte offset of the int32 [H_kv][n_ct] slot counts in `bytes`
};

// Latent rank tiles the busiest wave of a block accumulates (projection or value pass).
int max_owned(const BlockMeta& m) {
  const int nrt_k = m.rk_pad / 32, nrt_v = m.rv_pad / 32;
  const int ng = kWaves / v_segments(nrt_v);
  return std::max((nrt_k + kWaves - 1) / kWaves, (nrt_v + ng - 1) / ng);
}

int build_schedule(const milo_cache& c, const int32_t* table, int n_sel, const std::vector<int32_t>& tl, int n_ct,
                   Schedule* out) {
  const int NK = c.d / 16;
  auto item_cost = [&](const BlockMeta& m, int nt) {
    const int nrt_k = m.rk_pad / 32, nks = m.rk_pad / 16, nrt_v = m.rv_pad / 32;
    const int nseg = v_segments(nrt_v), ng = kWaves / nseg;
    const int mk = (nrt_k + kWaves - 1) / kWaves, mv = (nrt_v + ng - 1) / ng;
    int rounds = 0;
    for (int h = nseg; h > 1; h /= 2) ++rounds;
    const double item_frags = (double)NK * mk + m.rv_pad / 32.0;
    const double tile_frags = nt * ((double)nks + 16.0 / nseg * mv);
    return kCostFragItem * item_frags + kCostFragTile * tile_frags + kCostTile * nt + kCostItem +
           kCostSegRound * rounds;
  };
  int S_kv = 1;
  while (S_kv < c.n_kv && S_kv < 32) S_kv *= 2;
  int C = 1;
  while (n_ct % (2 * C) == 0 && S_kv * 2 * C <= 32) C *= 2;
  const int S = S_kv * C;
  const int n_hc = (c.n_kv + S_kv - 1) / S_kv;
  const int n_cg = n_ct / C;  // column-tile groups
  const int n_gangs = kCUs / S;
  double total = 0.0;
  for (int j = 0; j < n_sel; ++j) {
    const BlockMeta& m = c.meta[table[j]];
    total += item_cost(m, m.T_pad / kTile) * n_cg * n_hc;
  }
  for (int32_t len : tl)
    total += kCostTail * ((len + kTailChunk * C - 1) / (kTailChunk * C)) * n_hc;
  struct Part { int b, tile0, ntile; double cost; };
  struct Job { int part, req, ch, ct, hc; double cost; };
  // Jobs for one way of splitting the blocks: parts of at most `share` of a
  // gang's average work (and at most kMaxPartTiles tiles), longest first.
  auto make_jobs = [&](double share, std::vector<Part>& parts, std::vector<Job>& jobs) {
    const double target = std::max(1e-9, total / n_gangs * share);
    parts.clear();
    jobs.clear();
    for (int j = 0; j < n_sel; ++j) {
      const int b = table[j];
      const BlockMeta& m = c.meta[b];
      const int nt = m.T_pad / kTile;
      const int np_cost = (int)std::min<double>(nt, std::max(1.0, std::ceil(item_cost(m, nt) / target)));
      const int np = std::max(np_cost, (nt + kMaxPartTiles - 1) / kMaxPartTiles);
      for (int p = 0; p < np; ++p) {
        const int t_a = (int)((int64_t)nt * p / np), t_b = (int)((int64_t)nt * (p + 1) / np);
        parts.push_back({b, t_a, t_b - t_a, item_cost(m, t_b - t_a)});
      }
    }
    for (int p = 0; p < (int)parts.size(); ++p)
      for (int cg = 0; cg < n_cg; ++cg)
        for (int hc = 0; hc < n_hc; ++hc) jobs.push_back({p, -1, -1, cg, hc, parts[p].cost});
    for (int i = 0; i < (int)tl.size(); ++i)
      for (int chg = 0; chg * C * kTailChunk < tl[i]; ++chg)
        for (int hc = 0; hc < n_hc; ++hc) jobs.push_back({-1, i, chg, 0, hc, kCostTail});
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
    for (auto& l : lists)  // tail jobs first, then the longest block jobs
      std::stable_sort(l.begin(), l.end(), [&](int x, int y) {
        if ((jobs[x].part < 0) != (jobs[y].part < 0)) return jobs[x].part < 0;
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
    out->rk_pad_max = std::max(out->rk_pad_max, c.meta[pt.b].rk_pad);
    out->rv_pad_max = std::max(out->rv_pad_max, c.meta[pt.b].rv_pad);
    out->max_own = std::max(out->max_own, max_owned(c.meta[pt.b]));
  }

  // a workgroup folds consecutive block items of one (KV head, column tile)
  // into one partial where the kernel keeps that partial in registers (at most
  // two latent rank tiles per wave)
  const bool fold = out->max_own <= 2;
  // LDS plan: the projected query, weight tile and a 6-slot fragment ring,
  // the rest for the program (fewer launches would cost the ring); when even a
  // short program leaves no room for that (ranks above 512), the weight tile
  // in two 128-token halves and a 4-slot ring; failing that, no ring
  const size_t short_prog = 16 * sizeof(WorkItem) + (size_t)kWaves * kRunBufs * kRunCap * sizeof(int2);
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
  if (const int64_t pc = env_program_cap(); pc >= 0) cap = std::min(cap, (size_t)pc);
  for (int L = 1; L <= (1 << 20); L *= 2) {
    std::vector<std::vector<unsigned char>> progs((size_t)L * kCUs);
    std::vector<WgProgram> entries((size_t)L * kCUs);
    std::vector<int32_t> slot_count((size_t)c.n_kv * n_ct, 0);
    size_t max_prog = 0;
    for (int l = 0; l < L; ++l) {
      std::vector<int> idx;
      for (size_t k = l; k < jobs.size(); k += L) idx.push_back((int)k);
      std::vector<std::vector<int>> lists;
      deal(jobs, idx, lists);
      for (int gang = 0; gang < n_gangs; ++gang) {
        for (int j = 0; j < S; ++j) {
          const int wg = (gang % kXcds) + kXcds * ((gang / kXcds) * S + j);
          std::vector<WorkItem> items;
          const int sub = j / S_kv;  // column tile (or tail chunk) within the job's group
          for (int k : lists[gang]) {
            const Job& jb = jobs[k];
            const int g = jb.hc * S_kv + j % S_kv;
            if (g >= c.n_kv) continue;
            WorkItem w{};
            w.g = g;
            if (jb.part >= 0) {
              const Part& pt = parts[jb.part];
              w.blk = c.meta[pt.b];
              w.kind = kItemBlock;
              w.slot = jb.part;
              w.sub = jb.ct * C + sub;
              w.tile0 = pt.tile0;
              w.ntile = pt.ntile;
              w.flags = lg_rank_groups(w.blk.rv_pad / 32) << kItemLgNgShift;
            } else {
              const int ch = jb.ch * C + sub;
              if (ch * kTailChunk >= tl[jb.req]) continue;
              w.kind = kItemTail;
              w.blk.T = std::min(kTailChunk, tl[jb.req] - ch * kTailChunk);  // tokens of the chunk
              w.req = jb.req;
              w.slot = ch;
              w.sub = ch;
            }
            items.push_back(w);
          }
          // groups of consecutive block items with one (KV head, column tile)
          // share a slot; slots of a (head, tile) are numbered densely
          int first = -1, last = -1;
          for (int i = 0; i < (int)items.size(); ++i) {
            WorkItem& w = items[i];
            if (w.kind != kItemBlock) continue;
            const bool cont = fold && first >= 0 && items[first].g == w.g && items[first].sub == w.sub;
            if (cont) {
              w.slot = items[first].slot;
            } else {
              if (last >= 0) items[last].flags |= kItemFlush;
              first = i;
              w.flags |= kItemFirst;
              w.slot = slot_count[(size_t)w.g * n_ct + w.sub]++;
            }
            last = i;
          }
          if (last >= 0) items[last].flags |= kItemFlush;
          WgProgram& e = entries[(size_t)l * kCUs + wg];
          e = WgProgram{};
          if (items.empty()) continue;
          std::vector<unsigned char>& pb = progs[(size_t)l * kCUs + wg];
          pb.resize(items.size() * sizeof(WorkItem));
          std::memcpy(pb.data(), items.data(), pb.size());
          e.n_items = (int32_t)items.size();
          e.words = (int32_t)(pb.size() / 4);
          // LDS: the items, then every wave's run buffer
          max_prog = std::max(max_prog, pb.size() + (size_t)kWaves * kRunBufs * kRunCap * sizeof(int2));
        }
      }
    }
    const size_t prog_bytes = (size_t)round_up((int64_t)max_prog, 256);
    if (prog_bytes > cap) continue;
    // assemble: the entry table, every program at a 16-byte aligned offset,
    // then the slot counts
    size_t off = entries.size() * sizeof(WgProgram);
    for (size_t k = 0; k < progs.size(); ++k) {
      entries[k].off = (int64_t)off;
      off += progs[k].size();
    }
    out->count_off = (int64_t)round_up((int64_t)off, 16);
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
    return MILO_OK;
  }
  return fail(MILO_ERR_UNSUPPORTED, "work schedule does not fit in LDS");
}

void destroy(milo_cache* c) {
  if (!c) return;
  if (c->device >= 0) {
    int cur = -1;
    if (hipGetDevice(&cur) == hipSuccess && cur != c->device) (void)hipSetDevice(c->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(c->data);
    (void)hipFree(c->part_o);
    (void)hipFree(c->part_ml);
    (void)hipFree(c->plan_d);
    (void)hipFree(c->tail_len_d);
    (void)hipHostFree(c->plan_pinned);
    (void)hipHostFree(c->tail_len_pinned);
    if (cur >= 0 && cur != c->device) (void)hipSetDevice(cur);
  }
  delete c;
}

}  // namespace

namespace milo {
void clear_error() { g_err.clear(); }
int report_error(int code, const char* msg) { return fail(code, "%s", msg); }
bool timing_enabled() {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  return g_timing.enabled;
}
}  // namespace milo

extern "C" {

const char* milo_last_error(void) { return g_err.c_str(); }

int milo_cache_create(const milo_cache_desc* desc, const uint16_t* const* pk, const uint16_t* const* rk,
                      const uint16_t* const* pv, const uint16_t* const* rv, int src_on_device,
                      void* hip_stream, milo_cache** out) {
  g_err.clear();
  if (!out) return fail(MILO_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!desc) return fail(MILO_ERR_INVALID_ARG, "desc is NULL");
  if (desc->n_blocks < 1) return fail(MILO_ERR_INVALID_ARG, "n_blocks must be >= 1 (got %d)", desc->n_blocks);
  if (desc->n_kv_heads < 1) return fail(MILO_ERR_INVALID_ARG, "n_kv_heads must be >= 1");
  if (desc->head_dim != 64 && desc->head_dim != 128)
    return fail(MILO_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", desc->head_dim);
  if (!desc->block_tokens || !desc->rank_k || !desc->rank_v)
    return fail(MILO_ERR_INVALID_ARG, "block_tokens / rank_k / rank_v must be non-NULL");
  if (!pk || !rk || !pv || !rv) return fail(MILO_ERR_INVALID_ARG, "factor pointer arrays must be non-NULL");
  if (src_on_device != 0 && src_on_device != 1) return fail(MILO_ERR_INVALID_ARG, "src_on_device must be 0 or 1");
  const int64_t D = (int64_t)desc->n_kv_heads * desc->head_dim;
  for (int b = 0; b < desc->n_blocks; ++b) {
    const int T = desc->block_tokens[b], a = desc->rank_k[b], v = desc->rank_v[b];
    if (T < 1) return fail(MILO_ERR_INVALID_ARG, "block %d: T_b must be >= 1 (got %d)", b, T);
    if (a < 1 || a > T || a > D || v < 1 || v > T || v > D)
      return fail(MILO_ERR_INVALID_ARG, "block %d: ranks (%d, %d) must lie in [1, min(T_b=%d, H_kv*d=%lld)]",
                  b, a, v, T, (long long)D);
    if (a > kMaxRank || v > kMaxRank)
      return fail(MILO_ERR_UNSUPPORTED, "block %d: rank above the supported maximum %d", b, kMaxRank);
    if (!pk[b] || !rk[b] || !pv[b] || !rv[b]) return fail(MILO_ERR_INVALID_ARG, "block %d: NULL factor", b);
  }

  milo_cache* c = new milo_cache();
  c->n_blocks = desc->n_blocks;
  c->n_kv = desc->n_kv_heads;
  c->d = desc->head_dim;
  c->T.assign(desc->block_tokens, desc->block_tokens + c->n_blocks);
  c->rk.assign(desc->rank_k, desc->rank_k + c->n_blocks);
  c->rv.assign(desc->rank_v, desc->rank_v + c->n_blocks);
  c->meta.resize(c->n_blocks);
  int64_t off = 0, max_src = 0;
  for (int b = 0; b < c->n_blocks; ++b) {
    BlockMeta& m = c->meta[b];
    m.T = c->T[b];
    m.T_pad = (int)round_up(c->T[b], kTile);
    m.rk_pad = (int)round_up(c->rk[b], 32);
    m.rv_pad = (int)round_up(c->rv[b], 32);
    int64_t* offs[4] = {&m.off_pk, &m.off_rk, &m.off_pv, &m.off_rv};
    for (int w = 0; w < 4; ++w) {
      const FactorGeom f = geom_of(*c, b, w);
      *offs[w] = off;
      off = round_up(off + frag_count(f) * kFragElems, kAlignElems);
      max_src = std::max<int64_t>(max_src, (int64_t)f.rows * f.cols);
    }
  }
  c->data_elems = off;
  if (off / kFragElems >= ((int64_t)1 << 31)) {
    delete c;
    return fail(MILO_ERR_UNSUPPORTED, "cache of %lld elements exceeds the 2^31-fragment index range", (long long)off);
  }
  const int64_t need = off * 2 + (src_on_device ? 0 : max_src * 2);
  const int64_t cap = env_byte_cap();
  if (cap >= 0 && need > cap) {
    delete c;
    return fail(MILO_ERR_OUT_OF_MEMORY, "cache needs %lld device bytes, above MILO_MAX_DEVICE_BYTES=%lld",
                (long long)need, (long long)cap);
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  uint16_t* staging = nullptr;
  auto cleanup_fail = [&](int code) {
    if (staging) (void)hipFree(staging);
    destroy(c);
    return code;
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) { c->device = -1; return cleanup_fail(hip_fail(e, "hipGetDevice")); }
  if ((e = hipMalloc(&c->data, (size_t)c->data_elems * 2)) != hipSuccess)
    return cleanup_fail(hip_fail(e, "hipMalloc(packed factors)"));
  if (!src_on_device && (e = hipMalloc(&staging, (size_t)max_src * 2)) != hipSuccess)
    return cleanup_fail(hip_fail(e, "hipMalloc(staging)"));
  const uint16_t* const* srcs[4] = {pk, rk, pv, rv};
  for (int b = 0; b < c->n_blocks; ++b) {
    for (int w = 0; w < 4; ++w) {
      const FactorGeom f = geom_of(*c, b, w);
      const uint16_t* src = srcs[w][b];
      if (!src_on_device) {
        if ((e = hipMemcpyAsync(staging, src, (size_t)f.rows * f.cols * 2, hipMemcpyHostToDevice, s)) != hipSuccess)
          return cleanup_fail(hip_fail(e, "hipMemcpyAsync(factor)"));
        src = staging;
      }
      PackArgs pa{src, c->data + factor_offset(c->meta[b], w), f, frag_count(f)};
      if ((e = launch_pack(pa, s)) != hipSuccess) return cleanup_fail(hip_fail(e, "pack kernel"));
    }
  }
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return cleanup_fail(hip_fail(e, "hipStreamSynchronize"));
  if (staging) (void)hipFree(staging);
  staging = nullptr;
  *out = c;
  return MILO_OK;
}

void milo_cache_free(milo_cache* cache) { destroy(cache); }

int milo_cache_device_bytes(const milo_cache* cache, int64_t* bytes) {
  g_err.clear();
  if (!cache || !bytes) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *bytes = cache->data_elems * 2;
  return MILO_OK;
}

int milo_cache_read_factor(const milo_cache* cache, int32_t block, int32_t which, uint16_t* dst) {
  g_err.clear();
  if (!cache || !dst) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  if (block < 0 || block >= cache->n_blocks) return fail(MILO_ERR_INVALID_ARG, "block %d out of range", block);
  if (which < 0 || which > 3) return fail(MILO_ERR_INVALID_ARG, "which must be 0..3");
  const FactorGeom f = geom_of(*cache, block, which);
  const int64_t n = frag_count(f) * kFragElems;
  std::vector<uint16_t> packed((size_t)n);
  MILO_HIP(hipMemcpy(packed.data(), cache->data + factor_offset(cache->meta[block], which), (size_t)n * 2,
                     hipMemcpyDeviceToHost));
  for (int64_t fr = 0; fr < frag_count(f); ++fr)
    for (int lane = 0; lane < 64; ++lane)
      for (int e = 0; e < 8; ++e) {
        int row, col;
        frag_source(f, fr, lane, e, &row, &col);
        if (row < f.rows && col < f.cols) dst[(int64_t)row * f.cols + col] = packed[(size_t)(fr * kFragElems + lane * 8 + e)];
      }
  return MILO_OK;
}

// Attention of n_q query tokens over the selected blocks plus their dense tails:
// query i reads tail rows [i * tail_stride, i * tail_stride + tail_len[i]) of
// tail_k / tail_v (tail_stride = tail_cap: one tail per request; 0: one shared tail).
static int attend(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_q, int32_t n_q_heads,
                  const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v, const int32_t* tail_len,
                  int32_t tail_cap, int64_t tail_stride, float scale, float* out, void* hip_stream) {
  // ---- validation (host only, nothing queued yet) ----
  if (!c) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  if (n_sel < 0) return fail(MILO_ERR_INVALID_ARG, "n_sel must be >= 0");
  if (n_sel > 0 && !block_table) return fail(MILO_ERR_INVALID_ARG, "block_table is NULL");
  if (n_q < 1) return fail(MILO_ERR_INVALID_ARG, "n_q must be >= 1");
  if (n_q_heads < 1 || n_q_heads % c->n_kv != 0)
    return fail(MILO_ERR_INVALID_ARG, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)", n_q_heads,
                c->n_kv);
  const int G = n_q_heads / c->n_kv;
  if (G > kMaxGroup) return fail(MILO_ERR_UNSUPPORTED, "more than %d query heads per KV head", kMaxGroup);
  if (!q || !out) return fail(MILO_ERR_INVALID_ARG, "q / out must be non-NULL");
  if (tail_cap < 0) return fail(MILO_ERR_INVALID_ARG, "tail_cap must be >= 0");
  if (tail_cap > 0 && (!tail_k || !tail_v || !tail_len))
    return fail(MILO_ERR_INVALID_ARG, "tail_k / tail_v / tail_len must be non-NULL when tail_cap > 0");
  if (!std::isfinite(scale)) return fail(MILO_ERR_INVALID_ARG, "scale must be finite");
  if ((int64_t)n_q * n_q_heads > (int64_t)1 << 24) return fail(MILO_ERR_UNSUPPORTED, "too many query columns");
  std::vector<int32_t> tl(n_q, 0);
  for (int i = 0; i < n_q; ++i) {
    if (tail_cap > 0) tl[i] = tail_len[i];
    if (tl[i] < 0 || tl[i] > tail_cap)
      return fail(MILO_ERR_INVALID_ARG, "tail_len[%d]=%d outside [0, tail_cap=%d]", i, tl[i], tail_cap);
    if (n_sel == 0 && tl[i] == 0) return fail(MILO_ERR_INVALID_ARG, "request %d has no keys to attend to", i);
  }
  if (n_sel > 0) {
    std::vector<char> seen(c->n_blocks, 0);
    for (int j = 0; j < n_sel; ++j) {
      const int b = block_table[j];
      if (b < 0 || b >= c->n_blocks)
        return fail(MILO_ERR_INVALID_ARG, "block_table[%d]=%d outside [0, %d)", j, b, c->n_blocks);
      if (seen[b]) return fail(MILO_ERR_INVALID_ARG, "block id %d selected twice", b);
      seen[b] = 1;
    }
  }
  int dev = -1;
  MILO_HIP(hipGetDevice(&dev));
  if (dev != c->device) return fail(MILO_ERR_INVALID_ARG, "cache lives on device %d, current device is %d", c->device, dev);
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);

  // ---- plan (rebuilt only when the call's shape changes) ----
  std::vector<int32_t> key;
  key.reserve(6 + n_sel + n_q);
  key.push_back(n_sel);
  key.push_back(n_q);
  key.push_back(n_q_heads);
  key.push_back(tail_cap);
  key.insert(key.end(), block_table, block_table + n_sel);
  key.insert(key.end(), tl.begin(), tl.end());
  const int n_cols = n_q * n_q_heads;
  int max_chunks = 0;
  for (int i = 0; i < n_q; ++i) max_chunks = std::max(max_chunks, (tl[i] + kTailChunk - 1) / kTailChunk);
  if (key != c->plan_key) {
    // no plan is valid until this one is complete: a failure below (an
    // allocation, an upload) must not leave the old key pointing at buffers
    // that were freed or half rewritten
    c->plan_key.clear();
    const int ncg = n_q * G;
    const int n_ct = (ncg + kCols - 1) / kCols;
    Schedule sch;
    const int err = build_schedule(*c, block_table, n_sel, tl, n_ct, &sch);
    if (err != MILO_OK) return err;
    const int max_rt = sch.max_own <= 2 ? 2 : sch.max_own == 3 ? 3 : 4;
    // deepest fragment ring that fits next to the program, projected query and
    // weight tile (4 slots go with the half weight tile)
    const size_t base = attend_lds_base_bytes(c->d, sch.rk_pad_max, sch.rv_pad_max, sch.half_w);
    const size_t prog = (size_t)sch.prog_bytes;
    int nslot = 0;
    if (sch.half_w) {
      // the program was sized to leave room for this ring
      if (prog + base + attend_ring_bytes(4) > (size_t)kLdsBytes)
        return fail(MILO_ERR_UNSUPPORTED, "work schedule does not fit in LDS");
      nslot = 4;
    } else {
      for (int cand : {8, 6})
        if (prog + base + attend_ring_bytes(cand) <= (size_t)kLdsBytes) { nslot = cand; break; }
    }
    // device buffers
    const int64_t plan_bytes = (int64_t)sch.bytes.size();
    if (plan_bytes > c->plan_cap) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->plan_d);
      (void)hipHostFree(c->plan_pinned);
      c->plan_d = nullptr;
      c->plan_pinned = nullptr;
      c->plan_cap = 0;
      MILO_HIP(hipMalloc(&c->plan_d, (size_t)plan_bytes));
      MILO_HIP(hipHostMalloc(&c->plan_pinned, (size_t)plan_bytes, hipHostMallocDefault));
      c->plan_cap = plan_bytes;
    }
    if (n_q > c->tail_len_cap) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->tail_len_d);
      (void)hipHostFree(c->tail_len_pinned);
      c->tail_len_d = nullptr;
      c->tail_len_pinned = nullptr;
      c->tail_len_cap = 0;
      MILO_HIP(hipMalloc(&c->tail_len_d, sizeof(int32_t) * n_q));
      MILO_HIP(hipHostMalloc(&c->tail_len_pinned, sizeof(int32_t) * n_q, hipHostMallocDefault));
      c->tail_len_cap = n_q;
    }
    // the pinned staging buffers may still feed an earlier upload
    MILO_HIP(hipStreamSynchronize(s));
    std::memcpy(c->plan_pinned, sch.bytes.data(), (size_t)plan_bytes);
    std::memcpy(c->tail_len_pinned, tl.data(), sizeof(int32_t) * n_q);
    MILO_HIP(hipMemcpyAsync(c->plan_d, c->plan_pinned, (size_t)plan_bytes, hipMemcpyHostToDevice, s));
    MILO_HIP(hipMemcpyAsync(c->tail_len_d, c->tail_len_pinned, sizeof(int32_t) * n_q, hipMemcpyHostToDevice, s));
    c->n_launch = sch.n_launch;
    c->n_slots = sch.n_block_slots + max_chunks;
    c->n_block_slots = sch.n_block_slots;
    c->count_off = sch.count_off;
    c->n_ct = n_ct;
    c->max_rt = max_rt;
    c->nslot = nslot;
    c->rk_pad_max = sch.rk_pad_max;
    c->prog_bytes = sch.prog_bytes;
    c->ring_offset = (int)base;
    c->lds = prog + base + attend_ring_bytes(nslot);
    c->plan_key.swap(key);
  }
  const int64_t need = (int64_t)n_cols * c->n_slots;
  if (need > c->part_cols_slots) {
    MILO_HIP(hipStreamSynchronize(s));
    (void)hipFree(c->part_o);
    (void)hipFree(c->part_ml);
    c->part_o = nullptr;
    c->part_ml = nullptr;
    c->part_cols_slots = 0;
    const int64_t cap = env_byte_cap();
    const int64_t bytes = need * ((int64_t)c->d * 4 + 8);
    if (cap >= 0 && c->data_elems * 2 + bytes > cap)
      return fail(MILO_ERR_OUT_OF_MEMORY, "workspace of %lld bytes exceeds MILO_MAX_DEVICE_BYTES", (long long)bytes);
    MILO_HIP(hipMalloc(&c->part_o, (size_t)need * c->d * 4));
    MILO_HIP(hipMalloc(&c->part_ml, (size_t)need * sizeof(float2)));
    c->part_cols_slots = need;
  }

  // ---- launches ----
  AttendArgs aa{};
  aa.data = c->data;
  aa.prog = c->plan_d;
  aa.q = q;
  aa.tail_k = tail_k;
  aa.tail_v = tail_v;
  aa.tail_len = c->tail_len_d;
  aa.part_o = c->part_o;
  aa.part_ml = c->part_ml;
  aa.qscale = scale * 1.4426950408889634f;
  aa.n_q = n_q;
  aa.H_q = n_q_heads;
  aa.H_kv = c->n_kv;
  aa.G = G;
  aa.tail_stride = tail_stride;
  aa.n_slots = c->n_slots;
  aa.n_block_slots = c->n_block_slots;
  aa.qt_stride = c->rk_pad_max + 8;
  aa.prog_bytes = c->prog_bytes;
  aa.ring_offset = c->ring_offset;
  MergeArgs ma{c->part_o, c->part_ml, c->tail_len_d, out,
               reinterpret_cast<const int32_t*>(c->plan_d + c->count_off), n_q_heads, G, c->n_ct,
               c->n_block_slots, c->n_slots};

  // timing: events recorded by the launches themselves at kernel start and end
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};  // attend start / end, merge start / end
  bool timed = false;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    if (g_timing.enabled) {
      for (int k = 0; k < 4; ++k) {
        if (g_timing.pool.empty()) {
          hipEvent_t e;
          const hipError_t ce = hipEventCreate(&e);
          if (ce != hipSuccess) {
            for (int j = 0; j < k; ++j) g_timing.pool.push_back(ev[j]);
            return hip_fail(ce, "hipEventCreate");
          }
          g_timing.pool.push_back(e);
        }
        ev[k] = g_timing.pool.back();
        g_timing.pool.pop_back();
      }
      timed = true;
    }
  }
  // a failed launch hands the call's events back to the pool
  auto launch_fail = [&](hipError_t err, const char* what) {
    if (timed) {
      std::lock_guard<std::mutex> lk(g_timing.mu);
      g_timing.pool.insert(g_timing.pool.end(), ev, ev + 4);
    }
    return hip_fail(err, what);
  };
  hipError_t e = hipSuccess;
  for (int l = 0; l < c->n_launch; ++l) {
    aa.wg = reinterpret_cast<const WgProgram*>(c->plan_d) + (size_t)l * kCUs;
    e = launch_attend(aa, c->d, c->max_rt, c->nslot, kCUs, c->lds, s, l == 0 ? ev[0] : nullptr,
                      l == c->n_launch - 1 ? ev[1] : nullptr);
    if (e != hipSuccess) return launch_fail(e, "attend kernel launch");
  }
  e = launch_merge(ma, c->d, n_cols, s, ev[2], ev[3]);
  if (e != hipSuccess) return launch_fail(e, "merge kernel launch");
  if (timed) {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    g_timing.recorded.insert(g_timing.recorded.end(), ev, ev + 4);
  }
  return MILO_OK;
}

int milo_attend_decode(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_q, int32_t n_q_heads,
                       const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v, const int32_t* tail_len,
                       int32_t tail_cap, float scale, float* out, void* hip_stream) {
  g_err.clear();
  return attend(c, block_table, n_sel, n_q, n_q_heads, q, tail_k, tail_v, tail_len, tail_cap, tail_cap, scale, out,
                hip_stream);
}

int milo_attend_prefill(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_tok, int32_t n_q_heads,
                        const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v, int32_t tail_base,
                        int32_t tail_cap, float scale, float* out, void* hip_stream) {
  g_err.clear();
  if (n_tok < 1) return fail(MILO_ERR_INVALID_ARG, "n_tok must be >= 1");
  if (tail_base < 0) return fail(MILO_ERR_INVALID_ARG, "tail_base must be >= 0");
  if ((int64_t)tail_base + n_tok > tail_cap)
    return fail(MILO_ERR_INVALID_ARG, "tail_cap (%d) must hold tail_base + n_tok = %lld rows", tail_cap,
                (long long)tail_base + n_tok);
  if (!tail_k || !tail_v) return fail(MILO_ERR_INVALID_ARG, "tail_k / tail_v must be non-NULL");
  // token j sees the tail_base rows before the chunk and the chunk's first j + 1 tokens
  std::vector<int32_t> tl(n_tok);
  for (int j = 0; j < n_tok; ++j) tl[j] = tail_base + j + 1;
  return attend(c, block_table, n_sel, n_tok, n_q_heads, q, tail_k, tail_v, tl.data(), tail_cap, 0, scale, out,
                hip_stream);
}

int milo_timing_enable(int enable) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.enabled = enable != 0;
  return MILO_OK;
}

int milo_timing_read(double* attend_kernel_ms, double* merge_kernel_ms, int64_t* n_calls) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double ta = 0.0, tm = 0.0;
  const size_t n = g_timing.recorded.size() / 4;
  for (size_t k = 0; k < n; ++k) {
    hipEvent_t* e = &g_timing.recorded[4 * k];
    MILO_HIP(hipEventSynchronize(e[3]));
    float a = 0.f, m = 0.f;
    MILO_HIP(hipEventElapsedTime(&a, e[0], e[1]));
    MILO_HIP(hipEventElapsedTime(&m, e[2], e[3]));
    ta += a;
    tm += m;
  }
  g_timing.pool.insert(g_timing.pool.end(), g_timing.recorded.begin(), g_timing.recorded.end());
  g_timing.recorded.clear();
  if (attend_kernel_ms) *attend_kernel_ms = ta;
  if (merge_kernel_ms) *merge_kernel_ms = tm;
  if (n_calls) *n_calls = (int64_t)n;
  return MILO_OK;
}


}  // extern "C"
