// Internal definitions shared by the host API and the gfx950 kernels:
// the packed factor layout, per-block metadata, task encoding and kernel
// argument blocks.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace milo {

// ---------------------------------------------------------------------------
// Packed layout.  Every factor is stored as a sequence of 1 KiB "fragments":
// 64 lanes x 8 bf16, exactly the per-lane operand of one
// v_mfma_f32_32x32x16_bf16 (R^V: of one v_mfma_f32_16x16x32_bf16), so one
// wave loads one fragment with one fully coalesced 16-byte load per lane.  Rows beyond T_b and ranks beyond r are
// stored as zeros (tokens padded to whole 256-token tiles, ranks to 32).
//
// Lane l = 32*c + m (c = lane group 0/1, m = 0..31), element e = 0..7.
//   P^K fragment (token sub-tile tau, rank step kap):
//       P^K[32*tau + m][16*kap + 8*c + e]                         (A: tokens x rank)
//   P^V fragment (token step sig, rank tile rho):
//       P^V[16*sig + 8*c + e][32*rho + m]                         (A: rank x tokens)
//   R^K fragment (KV head g, rank tile rho, d step kap):
//       R^K[32*rho + m][g*d + 16*kap + 8*c + e]                   (A: rank x d)
//   R^V fragment (KV head g, 16-dim slice ds, 32-rank step kap), lane l = 16*qq + n:
//       R^V[32*kap + 8*qq + e][g*d + 16*ds + n]                   (A: d x rank, 16x16x32)
//
// Fragment order follows the attention kernel's work split, so that every wave
// of a workgroup reads each factor as contiguous runs in the order it consumes
// it.  The kWaves waves split a 256-token tile for the scores: wave w owns token
// sub-tile tau = 8t + w of tile t.  For the projection, rank tiles are dealt
// round-robin over all waves (wave w owns rho = w + kWaves*j).  The latent
// value pass and the up-projection split the waves into nseg = v_segments(nrt)
// token segments times ng = kWaves / nseg rank groups: wave w works on token
// segment w / ng (256 / nseg tokens of every tile) and owns the rank tiles
// rho = (w % ng) + ng*j, so low-rank blocks still keep every wave busy.  The
// up-projection gives every wave a 16-dim slice of the output over all ranks.
//   P^K: [w][t][kap]
//   P^V: [rg][sig][j]                (group rg's run has owned_tiles(nrt, rg, ng) per sig)
//   R^K: [g][w][j][kap]
//   R^V: [g][ds][kap]
// ---------------------------------------------------------------------------
constexpr int kFragElems = 512;  // 64 lanes x 8 bf16
constexpr int kWaves = 8;        // waves per attention workgroup (two per SIMD)
constexpr int kTile = 256;       // tokens per attention tile
constexpr int kMaxOwn = 2;       // most latent rank tiles one wave accumulates (see v_segments)
enum FactorKind : int { kPK = 0, kRK = 1, kPV = 2, kRV = 3 };

// rank tiles dealt round-robin over n owners: how many owner w holds, and how
// many the owners before it hold
__host__ __device__ inline int owned_tiles(int nrt, int w, int n) {
  return nrt > w ? (nrt - w + n - 1) / n : 0;
}
__host__ __device__ inline int owned_before(int nrt, int w, int n) {
  // owners v < nrt % n hold one tile more than nrt / n
  return w * (nrt / n) + (w < nrt % n ? w : nrt % n);
}

// Token segments of the latent value pass for a block with nrt rank tiles of
// 32: the split (1, 2, 4 or 8 segments) with the least work for the busiest
// wave, ties going to fewer segments (fewer partial sums to combine), with no wave
// owning more than kMaxOwn rank tiles; past 8 * kMaxOwn rank tiles no split
// qualifies and the block uses one segment (every wave owns nrt / 8 tiles).
__host__ __device__ constexpr int v_segments(int nrt) {
  int best = 1, best_work = 1 << 30;
  for (int nseg = 1; nseg <= kWaves; nseg *= 2) {
    const int ng = kWaves / nseg;
    const int own = (nrt + ng - 1) / ng;
    if (own > kMaxOwn) continue;
    const int work = own * (kTile / nseg);
    if (work < best_work) {
      best_work = work;
      best = nseg;
    }
  }
  return best;
}

struct BlockMeta {
  int64_t off_pk, off_rk, off_pv, off_rv;
  int32_t T, T_pad, rk_pad, rv_pad;
};

// INT8 P factors (a cache option; Sec. 5.3 combines the low-rank cache with
// INT8 quantisation): P^K and P^V are stored as int8 codes c with one fp32
// scale per token row, P[t][k] = s_t c[t][k] (s_t = max_k |P[t][k]| / 127,
// c = round-to-nearest-even(P / s_t), both in fp32).  Codes keep the fragment
// order above at one byte per element (a fragment is 512 bytes: lane l's 8
// codes at bytes 8l..8l+7), so one 1 KiB unit of the fragment stream holds two
// consecutive fragments of a run.  Each block's scales follow its P^V codes
// as 256-byte units, one per (256-token tile t, wave w): the K scales of the
// wave's 32 score tokens 256t + 32w + m (m = 0..31), then their V scales.
constexpr int kScaleUnitBytes = 256;
// bytes of the int8 codes of a P factor with T_pad tokens and rank r_pad, and
// the offset (in bf16 elements of the cache buffer) of a block's scale units
__host__ __device__ inline int64_t i8_factor_bytes(int T_pad, int r_pad) { return (int64_t)T_pad * r_pad; }
__host__ __device__ inline int64_t i8_scale_offset(int64_t off_pv, int T_pad, int rv_pad) {
  return off_pv + i8_factor_bytes(T_pad, rv_pad) / 2;
}
__host__ __device__ inline int64_t i8_scale_bytes(int T_pad) { return (int64_t)(T_pad / kTile) * kWaves * kScaleUnitBytes; }

// Most 256-token tiles in one block item (parts of larger blocks are split),
// most KV heads one 64-column tile may span, and so the most fragment runs
// one item gives a wave (plus an end marker): the R^K and R^V runs of every
// head, per tile the P^K run, the scale unit (INT8) and the P^V run.  A plan
// sizes its run buffers for its own items (run_cap_for; kRunCap at most).
constexpr int kMaxPartTiles = 8;
constexpr int kMaxTileHeads = 4;
constexpr int kRunCap = 2 * kMaxTileHeads + 3 * kMaxPartTiles + 2;
__host__ __device__ inline int run_cap_for(int max_heads, int max_tiles, bool i8) {
  return 2 * max_heads + (i8 ? 3 : 2) * max_tiles + 2;
}
constexpr int kRunBufs = 4;  // run buffers per wave in the attention kernel
// A run (x, n) names n units of one kind, encoded in bits 28-29 of n:
//   kRunBf16   bf16 fragments x .. x+n-1 (1 KiB each)
//   kRunI8     int8 fragments x .. x+n-1 (512 bytes each, n even: n/2 units of two)
//   kRunScale  n scale units from byte 256 x
constexpr int kRunKindShift = 28;
constexpr int kRunCountMask = (1 << kRunKindShift) - 1;
enum RunKind : int { kRunBf16 = 0, kRunI8 = 1, kRunScale = 2 };

// log2 of the rank groups (kWaves / nseg) of a block with nrt V rank tiles
__host__ __device__ inline int lg_rank_groups(int nrt) {
  const int nseg = v_segments(nrt);
  return nseg == 1 ? 3 : nseg == 2 ? 2 : nseg == 4 ? 1 : 0;
}

// The fragment runs wave w consumes for a block item (block bm, the nh KV
// heads g0 .. g0+nh-1 whose query columns the item's column tile holds, tiles
// [tile0, tile0 + ntile)) of head dimension d, in the attention kernel's
// order: its R^K rank tiles of every head in turn (projection); then per tile
// its P^K sub-tile and the P^V rank tiles of its rank group over its token
// segment; then R^V for its 16-dim output slice over all ranks, every head in
// turn (up-projection).  lg_ng = lg_rank_groups(rv_pad / 32) (passed in, so
// the kernel derives runs with shifts only).  With INT8 P factors (i8) each
// tile's P^K and P^V runs are int8 runs and the wave's scale unit comes
// between them.  emit(first unit index, count | kind) is called for every
// non-empty run; offsets follow the packed layout above.
// A dense item (dense: a reconstructed block; bm = dense_meta of its head,
// offsets relative to the reconstruction buffer, frag_base fragments from the
// factor buffer) has no R^K or R^V runs.
template <typename Emit>
__host__ __device__ inline void block_runs(const BlockMeta& bm, int g0, int nh, int tile0, int ntile, int w, int d,
                                           int lg_ng, bool i8, Emit&& emit, bool dense = false, int frag_base = 0) {
  static_assert(kWaves == 8, "rank tiles are dealt over 8 waves");
  const int NK = d / 16;
  const int nrt_k = bm.rk_pad >> 5, nks = bm.rk_pad >> 4, nrt_v = bm.rv_pad >> 5;
  // owner w of tiles dealt round-robin over n = 2^lg owners: nrt >> lg tiles,
  // one more if w < nrt mod n; the owners before it hold w (nrt >> lg) + min(w, nrt mod n)
  const int own_k = (nrt_k >> 3) + (w < (nrt_k & 7) ? 1 : 0);
  const int before_k = w * (nrt_k >> 3) + (w < (nrt_k & 7) ? w : (nrt_k & 7));
  const int ng = 1 << lg_ng, rg = w & (ng - 1), sg = w >> lg_ng;
  const int rem_v = nrt_v & (ng - 1);
  const int own_v = (nrt_v >> lg_ng) + (rg < rem_v ? 1 : 0);
  const int before_v = rg * (nrt_v >> lg_ng) + (rg < rem_v ? rg : rem_v);
  const int nst = 2 << lg_ng;  // 16-token steps of a segment per tile (16 / nseg)
  const int tiles_all = bm.T_pad / kTile;
  // a dense item's offsets count from the reconstruction buffer; every other
  // item's from the factor buffer itself
  const int fb = dense ? frag_base : 0;
  const int rk0 = (int)(bm.off_rk / kFragElems), pk0 = (int)(bm.off_pk / kFragElems) + fb;
  const int pv0 = (int)(bm.off_pv / kFragElems) + fb, rv0 = (int)(bm.off_rv / kFragElems);
  if (own_k > 0 && !dense)
    for (int h = 0; h < nh; ++h) emit(rk0 + (g0 + h) * nrt_k * NK + NK * before_k, NK * own_k);
  const int pv_first = (bm.T_pad / 16) * before_v;
  if (i8) {
    // int8 fragment indices count 512-byte units from the buffer start
    const int pk8 = (int)(bm.off_pk / 256), pv8 = (int)(bm.off_pv / 256);
    const int sc0 = (int)(i8_scale_offset(bm.off_pv, bm.T_pad, bm.rv_pad) * 2 / kScaleUnitBytes);
    for (int t = tile0; t < tile0 + ntile; ++t) {
      emit(pk8 + (w * tiles_all + t) * nks, nks | (kRunI8 << kRunKindShift));
      emit(sc0 + t * kWaves + w, 1 | (kRunScale << kRunKindShift));
      if (own_v > 0) emit(pv8 + pv_first + (16 * t + nst * sg) * own_v, (nst * own_v) | (kRunI8 << kRunKindShift));
    }
  } else {
    for (int t = tile0; t < tile0 + ntile; ++t) {
      emit(pk0 + (w * tiles_all + t) * nks, nks);
      if (own_v > 0) emit(pv0 + pv_first + (16 * t + nst * sg) * own_v, nst * own_v);
    }
  }
  if (dense) return;
  const int nds = d / 16, nkr = bm.rv_pad >> 5;
  for (int h = 0; h < nh; ++h) emit(rv0 + ((g0 + h) * nds + w % nds) * nkr, nkr);
}

struct FactorGeom {
  int kind;
  int rows, cols;      // logical source shape (row-major, ld = cols)
  int T_pad, r_pad;    // padded token count (P) and padded rank
  int n_kv, d;         // for R factors
};

__host__ __device__ inline int64_t frag_count(const FactorGeom& f) {
  switch (f.kind) {
    case kPK: return (int64_t)(f.T_pad / 32) * (f.r_pad / 16);
    case kPV: return (int64_t)(f.T_pad / 16) * (f.r_pad / 32);
    case kRK: return (int64_t)f.n_kv * (f.r_pad / 32) * (f.d / 16);
    default:  return (int64_t)f.n_kv * (f.d / 16) * (f.r_pad / 32);
  }
}

// the owner whose run holds unit u, when owner w's run has per*owned_tiles(nrt, w, n)
// units and the runs are stored in owner order; *first = start of that run
__host__ __device__ inline int run_owner(int nrt, int64_t u, int64_t per, int n, int64_t* first) {
  int w = 0;
  int64_t start = 0;
  while (w + 1 < n && u >= start + per * owned_tiles(nrt, w, n)) {
    start += per * owned_tiles(nrt, w, n);
    ++w;
  }
  *first = start;
  return w;
}

// Source (row, col) of element e of lane `lane` in fragment `frag`.
__host__ __device__ inline void frag_source(const FactorGeom& f, int64_t frag, int lane, int e,
                                            int* row, int* col) {
  const int m = lane & 31, c = lane >> 5;
  switch (f.kind) {
    case kPK: {
      const int nks = f.r_pad / 16, ntiles = f.T_pad / kTile;
      const int kap = (int)(frag % nks);
      const int t = (int)((frag / nks) % ntiles);
      const int w = (int)(frag / ((int64_t)nks * ntiles));
      const int tau = kWaves * t + w;
      *row = 32 * tau + m;
      *col = 16 * kap + 8 * c + e;
      return;
    }
    case kPV: {
      const int nrt = f.r_pad / 32, T16 = f.T_pad / 16;
      const int ng = kWaves / v_segments(nrt);
      int64_t first;
      const int rg = run_owner(nrt, frag, T16, ng, &first);
      const int own = owned_tiles(nrt, rg, ng);
      const int64_t local = frag - first;
      const int sig = (int)(local / own), j = (int)(local % own);
      *row = 16 * sig + 8 * c + e;
      *col = 32 * (rg + ng * j) + m;
      return;
    }
    case kRK: {
      const int nk = f.d / 16, nrt = f.r_pad / 32;
      const int g = (int)(frag / ((int64_t)nrt * nk));
      const int64_t in_g = frag % ((int64_t)nrt * nk);
      int64_t first;
      const int w = run_owner(nrt, in_g, nk, kWaves, &first);
      const int64_t local = in_g - first;
      const int j = (int)(local / nk), kap = (int)(local % nk);
      *row = 32 * (w + kWaves * j) + m;
      *col = g * f.d + 16 * kap + 8 * c + e;
      return;
    }
    default: {
      const int nks = f.r_pad / 32, nds = f.d / 16;
      const int kap = (int)(frag % nks);
      const int ds = (int)((frag / nks) % nds);
      const int g = (int)(frag / ((int64_t)nks * nds));
      *row = 32 * kap + 8 * (lane >> 4) + e;
      *col = g * f.d + 16 * ds + (lane & 15);
      return;
    }
  }
}

// Fragment index (in 1 KiB units from the buffer start) of a given fragment of
// each factor of block bm, the inverse of frag_source for that factor:
//   P^K (token sub-tile tau, 16-rank step kap)     P^V (16-token step sig, rank tile rho)
//   R^K (KV head g, rank tile rho, 16-dim step kap) R^V (KV head g, 16-dim slice ds, 32-rank step kap)
__host__ __device__ inline int64_t pk_frag(const BlockMeta& bm, int tau, int kap) {
  const int nks = bm.rk_pad / 16, tiles_all = bm.T_pad / kTile;
  return bm.off_pk / kFragElems + ((int64_t)(tau % kWaves) * tiles_all + tau / kWaves) * nks + kap;
}
__host__ __device__ inline int64_t pv_frag(const BlockMeta& bm, int sig, int rho) {
  const int nrt = bm.rv_pad / 32, ng = kWaves / v_segments(nrt);
  const int rg = rho % ng, j = rho / ng;
  return bm.off_pv / kFragElems + (int64_t)(bm.T_pad / 16) * owned_before(nrt, rg, ng) +
         (int64_t)sig * owned_tiles(nrt, rg, ng) + j;
}
__host__ __device__ inline int64_t rk_frag(const BlockMeta& bm, int d, int g, int rho, int kap) {
  const int nk = d / 16, nrt = bm.rk_pad / 32;
  return bm.off_rk / kFragElems + (int64_t)g * nrt * nk + (int64_t)nk * (owned_before(nrt, rho % kWaves, kWaves) + rho / kWaves) +
         kap;
}
__host__ __device__ inline int64_t rv_frag(const BlockMeta& bm, int d, int g, int ds, int kap) {
  const int nds = d / 16, nkr = bm.rv_pad / 32;
  return bm.off_rv / kFragElems + ((int64_t)g * nds + ds) * nkr + kap;
}

// The same indices with the per-block splits precomputed, for inner loops:
// P^V with lg = lg_rank_groups(nrt) (rank groups ng = 2^lg) and T16 = T_pad / 16,
// R^K with nrt its 32-rank tiles and nk = d / 16 (pv0 / rk0: the factor's
// first fragment; rk_head: nrt * nk fragments per KV head).
__host__ __device__ inline int pv_frag_split(int pv0, int T16, int nrt, int lg, int sig, int rho) {
  const int ng = 1 << lg, rg = rho & (ng - 1), j = rho >> lg;
  const int q = nrt >> lg, rem = nrt & (ng - 1);
  const int before = rg * q + (rg < rem ? rg : rem), own = q + (rg < rem ? 1 : 0);
  return pv0 + T16 * before + sig * own + j;
}
__host__ __device__ inline int rk_frag_split(int rk0, int nrt, int nk, int g, int rho, int kap) {
  const int w = rho & (kWaves - 1), j = rho >> 3, q = nrt >> 3, rem = nrt & (kWaves - 1);
  static_assert(kWaves == 8, "rank tiles are dealt over 8 waves");
  return rk0 + g * nrt * nk + nk * (w * q + (w < rem ? w : rem) + j) + kap;
}

// ---------------------------------------------------------------------------
// Reconstruct-then-attend (Sec. 4.5 inference path, Alg. 1 full-rank
// reconstruction): a selected block may instead be rebuilt as its full-rank keys
// and values, K_b = P^K R^K and V_b = P^V R^V (fp32 accumulation; keys stored as
// fp16, values as bf16), into a
// per-call buffer, and then attended like an uncompressed block.  For KV head g
// the buffer holds K_{b,g} (T_pad x d) in the P^K fragment layout and V_{b,g}
// in the P^V fragment layout, both with "rank" d, so the attention kernel reads
// them with its latent loops unchanged: the scores of a column are K_{b,g} q
// (the query itself, as fp16, takes the place of the projected query; fp16
// score MFMAs, the scale on the fp32 scores) and the
// value pass yields the output directly (no up-projection).  Such "dense"
// block items need one KV head per column tile.
//   region of reconstructed block i: 2 T_pad D elements; head g at 2 g T_pad d,
//   its V at + T_pad d.
// The reconstruction kernel takes one task per (block, K or V, KV head, 256-token tile).
struct ReconBlock {
  BlockMeta src;    // the block's factors in the cache buffer
  int64_t dst;      // element offset of its region in the reconstruction buffer
  int32_t pos0;     // pre-RoPE keys: position of the block's first token; -1: keys as stored
  int32_t pad;
};
static_assert(sizeof(ReconBlock) == 64, "reconstruction block layout");
// task: x = reconstruction block (-1: none), y = tile << 8 | g << 1 | side (0: K, 1: V)
// Rotary embedding of pre-RoPE keys (Sec. 3: the factorised keys are taken
// before the rotation, which does not commute with R^K, so such blocks are
// reconstructed and rotated before attention).  Rotate-half arrangement: dim
// j < d/2 pairs with j + d/2 and the pair at position p turns by p w_j,
// w_j = theta^(-2j/d).  The kernel forms the angle in turns, p w_j / (2 pi),
// in fp64 from the table of w_j / (2 pi), keeps its fractional part and takes
// sine and cosine in fp32; positions are int32.
constexpr int64_t kRopeMaxEnd = 2147483647;  // every padded row's position below this
struct ReconArgs {
  const uint16_t* data;       // packed factors
  uint16_t* recon;            // reconstruction buffer
  const ReconBlock* blocks;   // [n_recon]
  const int2* tasks;          // [grid]
  const double* rope_turns;   // [d/2] w_j / (2 pi) of pre-RoPE keys (NULL: none)
};
// the BlockMeta of head g of a reconstructed block whose region starts at
// element `region` (offsets relative to the reconstruction buffer)
__host__ __device__ inline BlockMeta dense_meta(const BlockMeta& src, int64_t region, int g, int d) {
  BlockMeta m{};
  m.T = src.T;
  m.T_pad = src.T_pad;
  m.rk_pad = d;
  m.rv_pad = d;
  m.off_pk = region + (int64_t)g * 2 * src.T_pad * d;
  m.off_pv = m.off_pk + (int64_t)src.T_pad * d;
  m.off_rk = 0;
  m.off_rv = 0;
  return m;
}

// Per-block metadata in device memory; offsets are in bf16 elements from the
// start of the cache's packed buffer.

// Work item of the attention kernel.  Block items carry their block's metadata
// inline, so an item is self-contained.
enum ItemKind : int32_t { kItemBlock = 0, kItemTail = 1 };
//
// Query columns are numbered head-major: column c = g * N_g + i * G + (h mod G)
// of KV head g = h / G, request i, query head h (N_g = n_q * G columns per KV
// head).  A block item works on one column tile, a range of at most kCols
// consecutive columns that may span up to kMaxTileHeads KV heads.
struct WorkItem {
  BlockMeta blk;      // block items: the block's packed offsets and padded sizes
  int32_t kind;       // ItemKind
  int32_t slot;       // block items: the group's partial slot (see kItemFirst);
                      // tail items: chunk index (slot n_block_slots + slot)
  int32_t g;          // tail items: KV head; block items: first KV head of the column tile
  int32_t sub;        // block items: column tile index; tail items: kTailChunk-token chunk
  int32_t req;        // tail items: request index; block items: first column of the tile
  int32_t tile0;      // block items: first 256-token tile of the block covered
  int32_t ntile;      // block items: number of tiles covered
  int32_t flags;      // block items: kItemFirst / kItemFlush and the packed fields below
};
static_assert(sizeof(WorkItem) == 80, "work item layout");
// Consecutive block items of a workgroup for the same KV head and column tile
// form a group that shares one partial slot: the first item starts the
// workgroup's running (max, sum, output) per column, every item folds its own
// partial into it (log-sum-exp), and the last one writes it out.  Slots of a
// (head, column tile) are numbered densely from 0; tail items write slot
// n_block_slots + their chunk index.
// kItemInt8: INT8 P factors; kItemDense: a reconstructed block (its metadata
// names one KV head's K and V in the reconstruction buffer)
// kItemCausal: a dense item over a prefill chunk's shared tail, whose column of
// request i sees only its first tail_len_of(tl, i) tokens
enum ItemFlags : int32_t { kItemFirst = 1, kItemFlush = 2, kItemInt8 = 4, kItemDense = 8, kItemCausal = 16 };
// packed fields of a block item's flags: bits 8-9 lg_rank_groups of its block,
// bits 16-21 the tile's column count - 1, bits 24-26 its KV head count - 1
constexpr int kItemLgNgShift = 8;
constexpr int kItemColsShift = 16;
constexpr int kItemHeadsShift = 24;

// The attention kernel is persistent: workgroup b runs the program of entry b,
// a byte range of the program buffer holding its work items in order; it is
// copied into LDS at kernel start.  Each wave derives, item by item, the runs
// of consecutive packed fragments it consumes (a run is (first fragment index,
// count); block_runs below), into a per-wave run buffer of kRunCap entries
// that follows the items in LDS; after the last block item a sentinel run
// (fragment 0, 2^30) feeds the look-ahead loads issued past the last fragment.
struct WgProgram {
  int64_t off;                // byte offset in the program buffer (16-byte aligned)
  int32_t words;              // program size in 4-byte words
  int32_t n_items;            // work items (they start the program)
  int32_t pad[2];
};
static_assert(sizeof(WgProgram) == 24, "program entry layout");
constexpr int kSentinelRun = 1 << 27;  // a bf16 run long enough for any look-ahead

// Attention kernel geometry.
constexpr int kThreads = 64 * kWaves;
constexpr int kCols = 64;                      // query columns per workgroup
constexpr int kGemvCols = 16;                  // most columns of a tile whose projection may run as a GEMV
constexpr int kTokWave = kTile / kWaves;       // tokens per wave per tile (one MFMA row block)
static_assert(kTokWave == 32, "the score pass gives every wave one 32-token sub-tile");
constexpr int kWStride = kTile + 8;            // bf16 row stride of the weight tile in LDS
constexpr int kMaxGroup = 16;                  // max query heads per KV head
constexpr int kMaxRank = 896;                  // largest rank of the latent route (LDS bound)
constexpr int kMaxStoredRank = 1024;           // largest rank a cache stores (higher-rank blocks are reconstructed)
constexpr int kLdsBytes = 160 * 1024;          // LDS per workgroup on gfx950
constexpr int kTailChunk = kWaves * 32;        // dense-tail tokens per work item
constexpr int kXcds = 8;                       // XCDs of an MI355X (workgroup b runs on XCD b % 8)
constexpr int kCUs = 256;                      // compute units; one persistent workgroup each

// Per-request dense-tail lengths of one call, carried in the kernel arguments
// so that a call whose tails grew needs no upload: inline values (n_q <=
// kInlineTails), an affine rule base + step * i (the causal lengths of a
// prefill chunk, or no tails at all), or a device array for larger batches.
constexpr int kInlineTails = 256;
enum TailLenMode : int32_t { kTailInline = 0, kTailAffine = 1, kTailDevice = 2 };
struct TailLens {
  int32_t mode;
  int32_t base, step;        // kTailAffine: request i has base + step * i rows
  const int32_t* dev;        // kTailDevice: device [n_q]
  int32_t v[kInlineTails];   // kTailInline
};
__host__ __device__ inline int tail_len_of(const TailLens& t, int i) {
  return t.mode == kTailInline ? t.v[i] : t.mode == kTailAffine ? t.base + t.step * i : t.dev[i];
}

// How the head-major query columns are cut into column tiles:
//   kTilePacked  (N_g < kCols) every tile holds `a` whole KV heads
//   kTileHead    (N_g >= kCols) every KV head is cut into `a` tiles of kCols
//                columns, the last one partial
//   kTileFlat    (N_g >= kCols) tile t is columns [kCols t, kCols t + kCols),
//                spanning at most two KV heads
enum TileMode : int32_t { kTilePacked = 0, kTileHead = 1, kTileFlat = 2 };
struct TileGeom {
  int32_t mode, a, N_g, N;
};
// tile index of head-major column c, and the tile's first column and count
__host__ __device__ inline int tile_of(const TileGeom& t, int c) {
  return t.mode == kTilePacked ? (c / t.N_g) / t.a
         : t.mode == kTileHead ? (c / t.N_g) * t.a + (c % t.N_g) / kCols
                               : c / kCols;
}
__host__ __device__ inline void tile_range(const TileGeom& t, int tile, int* c0, int* cn) {
  int lo, hi;
  if (t.mode == kTilePacked) {
    lo = tile * t.a * t.N_g;
    hi = lo + t.a * t.N_g;
  } else if (t.mode == kTileHead) {
    const int g = tile / t.a, k = tile % t.a;
    lo = g * t.N_g + kCols * k;
    hi = lo + kCols < (g + 1) * t.N_g ? lo + kCols : (g + 1) * t.N_g;
  } else {
    lo = kCols * tile;
    hi = lo + kCols;
  }
  if (hi > t.N) hi = t.N;
  *c0 = lo;
  *cn = hi - lo;
}

struct AttendArgs {
  const uint16_t* data;      // packed factors
  const unsigned char* prog; // program buffer
  const WgProgram* wg;       // [grid] program of each workgroup
  const uint16_t* q;         // [n_q][H_q][d]
  const uint16_t* tail_k;    // request i's tail rows start at row i * tail_stride; [row][H_kv][d]
  const uint16_t* tail_v;
  float* part_o;             // [n_q*H_q][n_slots][d]
  float2* part_ml;           // [n_q*H_q][n_slots] (max in log2 units, sum)
  float qscale;              // scale * log2(e)
  int n_q, H_q, H_kv, G;
  int64_t tail_stride;      // rows between consecutive requests' tails (0: one tail shared by all)
  int n_slots;
  int n_block_slots;         // slots [0, n_block_slots) hold block groups, the rest tail chunks
  int qt_stride;             // bf16 row stride of the projected query in LDS
  int prog_bytes;            // LDS bytes reserved for the program (the work area follows)
  int ring_offset;           // byte offset of the per-wave fragment rings in the work area
  int N_g;                   // query columns per KV head, n_q * G
  int recon_delta;           // fragments from `data` to the reconstruction buffer (dense items)
  int run_cap;               // entries of a run buffer (the plan's bound, <= kRunCap)
  TailLens tl;               // tail lengths of this call
};

struct MergeArgs {
  const float* part_o;
  const float2* part_ml;
  float* out;                 // [n_q][H_q][d]
  const int32_t* slot_count;  // device [n_ct]: block-group slots used per column tile
  int H_q, G, n_block_slots, n_slots;
  TileGeom tiles;
  TailLens tl;
};

struct PackArgs {
  const uint16_t* src;
  uint16_t* dst;
  FactorGeom geom;
  int64_t n_frags;
  const float* row_scale;  // INT8 P factors: per-token scales [T_pad] (NULL: bf16)
};

// Launchers (defined in milo_kernels.hip).
// Host-side state shared by the library's entry points (defined with the
// decode entry points): the calling thread's error message and the timing flag.
void clear_error();
int report_error(int code, const char* msg);  // stores msg, returns code
bool timing_enabled();

hipError_t launch_pack(const PackArgs& a, hipStream_t s);
// bf16 factors in one launch: jobs and starts (n_jobs + 1 running sums of the
// jobs' fragment counts, n_frags = starts[n_jobs] - starts[0]) in device memory.
hipError_t launch_pack_batch(const PackArgs* jobs, const int64_t* starts, int n_jobs, int64_t n_frags,
                             hipStream_t s);
// INT8 P factors: per-row scales of a row-major bf16 factor [rows][cols] into
// scale[0 .. rows_pad) (rows past `rows` get 0); a row that is not finite sets *bad.
hipError_t launch_row_scales(const uint16_t* src, int rows, int cols, int rows_pad, float* scale, int* bad,
                             hipStream_t s);
// INT8 P factors: the scale units of a block from its K and V row scales
hipError_t launch_scale_units(const float* ks, const float* vs, int T_pad, float* dst, hipStream_t s);
// e0 / e1 (may be null): events recorded when the kernel starts and ends
// (hipExtLaunchKernelGGL), so they time the kernel itself.
// gemv: the kernel variant whose latent projection is a wavefront GEMV (tiles
// of at most kGemvCols columns; bf16 P factors only)
hipError_t launch_attend(const AttendArgs& a, int head_dim, int max_rt, int nslot, bool p_int8, bool gemv, int grid,
                         size_t lds_bytes, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_merge(const MergeArgs& a, int head_dim, int n_cols, hipStream_t s, hipEvent_t e0 = nullptr,
                        hipEvent_t e1 = nullptr);
// The shared tail of a prefill chunk (rows [0, rows) of tail_k / tail_v,
// [tail_cap][n_kv][d]) packed like a reconstructed block of T_pad tokens (rows
// past `rows` zero) at element `region` of the reconstruction buffer.
struct TailPackArgs {
  const uint16_t* tail_k;
  const uint16_t* tail_v;
  uint16_t* recon;
  int64_t region;
  int rows, T_pad, n_kv;
};
hipError_t launch_pack_tail(const TailPackArgs& a, int head_dim, hipStream_t s);
// Reconstruction of the dense blocks of a call: one workgroup per task.
hipError_t launch_recon(const ReconArgs& a, int head_dim, int n_tasks, hipStream_t s, hipEvent_t e0 = nullptr,
                        hipEvent_t e1 = nullptr);
// LDS of the attention kernel: a base region (projected query, weight tile and
// reductions, or the tail item's buffers) followed by kWaves rings of nslot fragments.
size_t attend_lds_base_bytes(int head_dim, int rk_pad_max, int rv_pad_max, bool half_w);
size_t attend_ring_bytes(int nslot);

}  // namespace milo
