// Work plan of one attention call (host only): how the query columns are cut
// into column tiles, and which work items every persistent workgroup of the
// attention kernel runs (programs in the kernel's WorkItem format).
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "milo_internal.h"

namespace milo {

// What the planner needs to know about a cache.
struct PlanInput {
  const BlockMeta* meta;  // [n_blocks]
  int n_kv, d;
  bool p_int8;            // P factors stored as INT8 codes (block items carry kItemInt8)
  // reconstruct-then-attend: per block id, the element offset of its region in
  // the reconstruction buffer, or -1 (latent); NULL: every block latent.  A plan
  // with reconstructed blocks needs one KV head per column tile.
  const int64_t* recon_region = nullptr;
  // a prefill chunk's shared tail, attended as a packed dense block: its block
  // id in meta / recon_region (its items carry kItemCausal), or -1
  int causal_block = -1;
};

struct Tiling {
  TileGeom geom{};
  int n_ct = 0;
  std::vector<int> c0, cn, g0, nh;  // per tile: first column, columns, first KV head, KV heads
};

int gang_size(int n_ct);
// head_tiles: one KV head per column tile (kTileHead), as dense items need;
// max_cols: most columns of a tile that packs whole KV heads (kGemvCols when
// the projection runs as a GEMV)
Tiling make_tiling(int n_kv, int N_g, bool head_tiles = false, int max_cols = kCols);

struct Schedule {
  std::vector<unsigned char> bytes;  // WgProgram[n_launch * kCUs], then the programs, then slot counts
  int n_launch = 0, n_parts = 0, prog_bytes = 0, rk_pad_max = 32, rv_pad_max = 32, max_own = 1;
  int n_block_slots = 0;  // block-group slots of the busiest column tile
  int gang = 1;           // workgroups per gang
  bool half_w = false;    // the weight tile in 128-token halves (LDS is short)
  int64_t count_off = 0;  // byte offset of the int32 [n_ct] slot counts in `bytes`
  int run_cap = kRunCap;  // entries of each wave's run buffers (run_cap_for of this plan's items)
};

int max_owned(const BlockMeta& m);

// The reconstruction work of a plan: the reconstructed blocks of the table (in
// table order) with their regions, and one task per (block, K or V, KV head,
// 256-token tile), ordered so that all tasks of one block's K (or V) run on one
// XCD (workgroup i runs on XCD i % 8; blocks dealt to the least loaded XCD),
// where they share the block's P and R factors in that XCD's L2.  Padding
// tasks (x = -1) fill the XCD queues to equal length.
struct ReconPlan {
  std::vector<ReconBlock> blocks;
  std::vector<int2> tasks;
  int64_t elems = 0;  // reconstruction buffer size (bf16 elements)
};
// Regions of the blocks table[0 .. n_sel) chosen by recon[j] != 0, laid out
// consecutively; fills region[block id] (others -1) and the tasks.  rope_pos
// (indexed by block id, or NULL): first-token positions of pre-RoPE keys.
void build_recon_plan(const BlockMeta* meta, const int32_t* table, int n_sel, const char* recon, int n_kv, int d,
                      std::vector<int64_t>* region, ReconPlan* out, const int32_t* rope_pos = nullptr);

// Build the plan for the selected blocks table[0 .. n_sel), n_q requests with
// n_chunks planned tail chunks each, over the column tiles `til`.  program_cap
// (< 0: none) caps the LDS bytes of a workgroup program.  Returns false with a
// message in *err when no plan fits.
bool build_schedule(const PlanInput& c, const int32_t* table, int n_sel, int n_q, int n_chunks, const Tiling& til,
                    int64_t program_cap, Schedule* out, std::string* err);

}  // namespace milo
