// Host-only check of the packed fragment layout declared in milo_internal.h:
// for each geometry given on the command line, every element of the padded
// source block is produced by exactly one (fragment, lane, element) and every
// (fragment, lane, element) maps inside the padded block.
#include <cstdio>
#include <cstdlib>
#include <string>
#include <utility>
#include <vector>

#include "milo_internal.h"

using namespace milo;

static int check(int kind, int T, int r, int n_kv, int d) {
  const int T_pad = (T + kTile - 1) / kTile * kTile;
  const int r_pad = (r + 31) / 32 * 32;
  FactorGeom f{};
  f.kind = kind;
  f.T_pad = T_pad;
  f.r_pad = r_pad;
  f.n_kv = n_kv;
  f.d = d;
  const int D = n_kv * d;
  int prow, pcol;  // padded source extent
  switch (kind) {
    case kPK: prow = T_pad; pcol = r_pad; break;
    case kPV: prow = T_pad; pcol = r_pad; break;
    default: prow = r_pad; pcol = D; break;
  }
  std::vector<int> seen((size_t)prow * pcol, 0);
  const long long nf = frag_count(f);
  if (nf * kFragElems != (long long)prow * pcol) {
    std::printf("kind %d: fragment count %lld does not cover %d x %d\n", kind, nf, prow, pcol);
    return 1;
  }
  for (long long fr = 0; fr < nf; ++fr)
    for (int lane = 0; lane < 64; ++lane)
      for (int e = 0; e < 8; ++e) {
        int row, col;
        frag_source(f, fr, lane, e, &row, &col);
        if (row < 0 || row >= prow || col < 0 || col >= pcol) {
          std::printf("kind %d: frag %lld lane %d e %d -> (%d, %d) outside %d x %d\n", kind, fr, lane, e, row, col,
                      prow, pcol);
          return 1;
        }
        seen[(size_t)row * pcol + col]++;
      }
  for (size_t k = 0; k < seen.size(); ++k)
    if (seen[k] != 1) {
      std::printf("kind %d: element (%zu, %zu) produced %d times\n", kind, k / pcol, k % pcol, seen[k]);
      return 1;
    }
  // the fragment index helpers (pk_frag, pv_frag, rk_frag, rv_frag) invert
  // frag_source: the coordinates of a fragment's lane 0, element 0 lead back to it
  BlockMeta bm{};
  bm.T = T;
  bm.T_pad = T_pad;
  bm.rk_pad = r_pad;
  bm.rv_pad = r_pad;
  for (long long fr = 0; fr < nf; ++fr) {
    int row, col;
    frag_source(f, fr, 0, 0, &row, &col);
    long long back;
    switch (kind) {
      case kPK: back = pk_frag(bm, row / 32, col / 16); break;
      case kPV: back = pv_frag(bm, row / 16, col / 32); break;
      case kRK: back = rk_frag(bm, d, col / d, row / 32, (col % d) / 16); break;
      default: back = rv_frag(bm, d, col / d, (col % d) / 16, row / 32); break;
    }
    if (back != fr) {
      std::printf("kind %d: fragment %lld starts at (%d, %d), whose index helper gives %lld\n", kind, fr, row, col,
                  back);
      return 1;
    }
    // the split forms of the reconstruction kernel's inner loop agree
    long long split = back;
    if (kind == kPV) split = pv_frag_split(0, T_pad / 16, r_pad / 32, lg_rank_groups(r_pad / 32), row / 16, col / 32);
    if (kind == kRK) split = rk_frag_split(0, r_pad / 32, d / 16, col / d, row / 32, (col % d) / 16);
    if (split != fr) {
      std::printf("kind %d: fragment %lld, split index form gives %lld\n", kind, fr, split);
      return 1;
    }
  }
  return 0;
}

// The fragment runs every wave derives for one whole block (block_runs), for a
// column tile of one KV head and for tiles spanning several heads: over the
// eight waves, each fragment of P^K, P^V and of the tile's heads' slices of R^K
// and R^V is read the expected number of times (once; R^V once per wave
// sharing a 16-dim slice), and each wave's run lengths match what the kernel
// consumes per phase.
static int check_runs(int T, int rk, int rv, int n_kv, int d) {
  const int T_pad = (T + kTile - 1) / kTile * kTile;
  BlockMeta bm{};
  bm.T = T;
  bm.T_pad = T_pad;
  bm.rk_pad = (rk + 31) / 32 * 32;
  bm.rv_pad = (rv + 31) / 32 * 32;
  const long long n_pk = (long long)T_pad * bm.rk_pad / kFragElems, n_pv = (long long)T_pad * bm.rv_pad / kFragElems;
  const long long n_rk = (long long)bm.rk_pad * n_kv * d / kFragElems, n_rv = (long long)bm.rv_pad * n_kv * d / kFragElems;
  bm.off_pk = 0;
  bm.off_rk = n_pk * kFragElems;
  bm.off_pv = (n_pk + n_rk) * kFragElems;
  bm.off_rv = (n_pk + n_rk + n_pv) * kFragElems;
  const long long total = n_pk + n_rk + n_pv + n_rv;
  const int ntile = T_pad / kTile, nds = d / 16;
  const int lg_ng = lg_rank_groups(bm.rv_pad / 32);
  // every head alone, and tiles spanning the heads g .. g + nh - 1
  const int nh_multi = n_kv < kMaxTileHeads ? n_kv : kMaxTileHeads;
  for (int pass = 0; pass < 2; ++pass)
  for (int g = 0; g + (pass ? nh_multi : 1) <= n_kv; ++g) {
    const int nh = pass ? nh_multi : 1;
    std::vector<int> seen((size_t)total, 0);
    for (int w = 0; w < kWaves; ++w) {
      std::vector<std::pair<int, int>> runs;
      block_runs(bm, g, nh, 0, ntile, w, d, lg_ng, false, [&](int x, int n) { runs.push_back({x, n}); });
      for (auto& r : runs)
        for (int k = 0; k < r.second; ++k) {
          if (r.first + k < 0 || r.first + k >= total) {
            std::printf("runs: fragment %d outside the block\n", r.first + k);
            return 1;
          }
          seen[(size_t)(r.first + k)]++;
        }
      // per-phase lengths the kernel takes
      const int nrt_k = bm.rk_pad / 32, nrt_v = bm.rv_pad / 32, nseg = v_segments(nrt_v), ng = kWaves / nseg;
      const int own_k = owned_tiles(nrt_k, w, kWaves), own_v = owned_tiles(nrt_v, w % ng, ng);
      size_t i = 0;
      for (int h = 0; h < nh; ++h)
        if (own_k > 0 && (runs[i++].second != d / 16 * own_k)) { std::printf("runs: R^K length\n"); return 1; }
      for (int t = 0; t < ntile; ++t) {
        if (runs[i++].second != bm.rk_pad / 16) { std::printf("runs: P^K length\n"); return 1; }
        if (own_v > 0 && runs[i++].second != kTile / 16 / nseg * own_v) { std::printf("runs: P^V length\n"); return 1; }
      }
      for (int h = 0; h < nh; ++h)
        if (runs[i++].second != bm.rv_pad / 32) { std::printf("runs: R^V length\n"); return 1; }
      if (i != runs.size()) { std::printf("runs: count\n"); return 1; }
      if ((int)runs.size() > kRunCap - 1) { std::printf("runs: more than the run buffer holds\n"); return 1; }
    }
    for (long long f = 0; f < total; ++f) {
      int want = 0;
      if (f < n_pk) want = 1;
      else if (f < n_pk + n_rk) {
        const long long h = (f - n_pk) / (n_rk / n_kv);
        want = h >= g && h < g + nh;
      } else if (f < n_pk + n_rk + n_pv) {
        want = 1;
      } else {
        const long long h = (f - n_pk - n_rk - n_pv) / (n_rv / n_kv);
        want = h >= g && h < g + nh ? kWaves / nds : 0;
      }
      if (seen[(size_t)f] != want) {
        std::printf("runs: head %d fragment %lld read %d times, want %d\n", g, f, seen[(size_t)f], want);
        return 1;
      }
    }
  }
  return 0;
}

// The same for INT8 P factors: over the eight waves every int8 fragment
// (512-byte unit) of P^K and P^V is read exactly once, every (tile, wave)
// scale unit exactly once and by that wave, between its P^K and P^V runs, and
// every int8 run has an even length (whole 1 KiB units of two fragments).
static int check_runs_i8(int T, int rk, int rv, int n_kv, int d) {
  const int T_pad = (T + kTile - 1) / kTile * kTile;
  BlockMeta bm{};
  bm.T = T;
  bm.T_pad = T_pad;
  bm.rk_pad = (rk + 31) / 32 * 32;
  bm.rv_pad = (rv + 31) / 32 * 32;
  const long long D = (long long)n_kv * d;
  // element offsets as the cache lays them out (each region on a 512-element boundary)
  auto up = [](long long x) { return (x + kFragElems - 1) / kFragElems * kFragElems; };
  bm.off_pk = 0;
  bm.off_rk = up(i8_factor_bytes(T_pad, bm.rk_pad) / 2);
  bm.off_pv = up(bm.off_rk + (long long)bm.rk_pad * D);
  bm.off_rv = up(bm.off_pv + i8_factor_bytes(T_pad, bm.rv_pad) / 2 + i8_scale_bytes(T_pad) / 2);
  const long long pk8_0 = bm.off_pk / 256, pk8_n = i8_factor_bytes(T_pad, bm.rk_pad) / 512;
  const long long pv8_0 = bm.off_pv / 256, pv8_n = i8_factor_bytes(T_pad, bm.rv_pad) / 512;
  const long long sc_0 = i8_scale_offset(bm.off_pv, T_pad, bm.rv_pad) * 2 / kScaleUnitBytes;
  const int ntile = T_pad / kTile, lg_ng = lg_rank_groups(bm.rv_pad / 32);
  std::vector<int> seen_pk(pk8_n, 0), seen_pv(pv8_n, 0), seen_sc(ntile * kWaves, 0);
  for (int w = 0; w < kWaves; ++w) {
    int last_kind = -1, tile = 0;
    bool bad = false;
    block_runs(bm, 0, 1, 0, ntile, w, d, lg_ng, true, [&](int x, int n) {
      const int kind = (n >> kRunKindShift) & 3, cnt = n & kRunCountMask;
      if (kind == kRunI8) {
        if (cnt % 2) bad = true;
        for (int k = 0; k < cnt; ++k) {
          const long long f = x + k;
          if (f >= pk8_0 && f < pk8_0 + pk8_n) seen_pk[f - pk8_0]++;
          else if (f >= pv8_0 && f < pv8_0 + pv8_n) seen_pv[f - pv8_0]++;
          else bad = true;
        }
      } else if (kind == kRunScale) {
        const long long u = x - sc_0;
        if (cnt != 1 || last_kind != kRunI8 || u != (long long)tile * kWaves + w) bad = true;
        else seen_sc[u]++;
        ++tile;
      }
      last_kind = kind;
    });
    if (bad) {
      std::printf("int8 runs: wave %d has a malformed run\n", w);
      return 1;
    }
  }
  for (auto* v : {&seen_pk, &seen_pv, &seen_sc})
    for (size_t k = 0; k < v->size(); ++k)
      if ((*v)[k] != 1) {
        std::printf("int8 runs: unit %zu read %d times\n", k, (*v)[k]);
        return 1;
      }
  return 0;
}

// Reconstructed blocks (dense items): for every KV head, the reconstruction
// kernel's stores (K_{b,g} as fragments (tau = 8 t + w, kap) holding dims
// 16 kap + 8 c + e of token 32 tau + m, V_{b,g} as fragments (sig = 16 t + s,
// rho) holding tokens 16 sig + 8 c + e of dim 32 rho + m) put every element of
// the head's region where frag_source says the P^K / P^V layouts of rank d
// keep it, each fragment exactly once; and the runs the eight waves derive for
// a dense item (offset by frag_base fragments) read each of those fragments
// once and nothing else (no R^K or R^V runs).
static int check_dense(int T, int n_kv, int d) {
  const int T_pad = (T + kTile - 1) / kTile * kTile, ntile = T_pad / kTile;
  BlockMeta src{};
  src.T = T;
  src.T_pad = T_pad;
  const int64_t region = 3 * (int64_t)kFragElems * 7;  // some region start (whole fragments)
  const int frag_base = -5;                            // buffer distance, in fragments
  const long long per_side = (long long)T_pad * d / kFragElems;
  for (int g = 0; g < n_kv; ++g) {
    const BlockMeta dm = dense_meta(src, region, g, d);
    const long long k0 = dm.off_pk / kFragElems, v0 = dm.off_pv / kFragElems;
    if (dm.off_pk % kFragElems || dm.off_pv != dm.off_pk + per_side * kFragElems ||
        dm.off_pk != region + 2LL * g * per_side * kFragElems) {
      std::printf("dense: head %d region offsets\n", g);
      return 1;
    }
    FactorGeom fk{}, fv{};
    fk.kind = kPK;
    fk.T_pad = T_pad;
    fk.r_pad = d;
    fv.kind = kPV;
    fv.T_pad = T_pad;
    fv.r_pad = d;
    std::vector<int> wk(per_side, 0), wv(per_side, 0);
    for (int t = 0; t < ntile; ++t)
      for (int f = 0; f < d / 2; ++f) {
        // K side store f: w = f / (d / 16), kap = f % (d / 16)
        {
          const int w = f / (d / 16), kap = f % (d / 16);
          const long long fr = pk_frag(dm, kWaves * t + w, kap) - k0;
          if (fr < 0 || fr >= per_side) { std::printf("dense: K store outside the region\n"); return 1; }
          wk[fr]++;
          for (int lane = 0; lane < 64; lane += 37)
            for (int e = 0; e < 8; e += 7) {
              int row, col;
              frag_source(fk, fr, lane, e, &row, &col);
              if (row != 32 * (kWaves * t + w) + (lane & 31) || col != 16 * kap + 8 * (lane >> 5) + e) {
                std::printf("dense: K fragment %lld lane %d e %d holds (%d, %d)\n", fr, lane, e, row, col);
                return 1;
              }
            }
        }
        // V side store f: s = f / (d / 32), rho = f % (d / 32)
        {
          const int sx = f / (d / 32), rho = f % (d / 32);
          const long long fr = pv_frag(dm, 16 * t + sx, rho) - v0;
          if (fr < 0 || fr >= per_side) { std::printf("dense: V store outside the region\n"); return 1; }
          wv[fr]++;
          for (int lane = 0; lane < 64; lane += 37)
            for (int e = 0; e < 8; e += 7) {
              int row, col;
              frag_source(fv, fr, lane, e, &row, &col);
              if (row != 16 * (16 * t + sx) + 8 * (lane >> 5) + e || col != 32 * rho + (lane & 31)) {
                std::printf("dense: V fragment %lld lane %d e %d holds (%d, %d)\n", fr, lane, e, row, col);
                return 1;
              }
            }
        }
      }
    for (long long k = 0; k < per_side; ++k)
      if (wk[k] != 1 || wv[k] != 1) {
        std::printf("dense: head %d fragment %lld stored %d / %d times\n", g, k, wk[k], wv[k]);
        return 1;
      }
    // the runs of a dense item over the whole block
    std::vector<int> rk_seen(per_side, 0), rv_seen(per_side, 0);
    for (int w = 0; w < kWaves; ++w) {
      int n_runs = 0;
      bool bad = false;
      block_runs(dm, g, 1, 0, ntile, w, d, lg_rank_groups(d / 32), false, [&](int x, int n) {
        ++n_runs;
        for (int k = 0; k < n; ++k) {
          const long long fr = (long long)x + k - frag_base;
          if (fr >= k0 && fr < k0 + per_side) rk_seen[fr - k0]++;
          else if (fr >= v0 && fr < v0 + per_side) rv_seen[fr - v0]++;
          else bad = true;
        }
      }, true, frag_base);
      if (bad || n_runs > 2 * ntile) {
        std::printf("dense: wave %d runs leave the head's region (%d runs)\n", w, n_runs);
        return 1;
      }
    }
    for (long long k = 0; k < per_side; ++k)
      if (rk_seen[k] != 1 || rv_seen[k] != 1) {
        std::printf("dense: head %d fragment %lld read %d / %d times\n", g, k, rk_seen[k], rv_seen[k]);
        return 1;
      }
  }
  return 0;
}

int main(int argc, char** argv) {
  if (argc > 1 && std::string(argv[1]) == "--dense") {
    int bad = 0, n = 0;
    for (int i = 2; i + 2 < argc; i += 3) {
      bad |= check_dense(std::atoi(argv[i]), std::atoi(argv[i + 1]), std::atoi(argv[i + 2]));
      ++n;
    }
    std::printf("%s (%d geometries)\n", bad ? "FAIL" : "OK", n);
    return bad;
  }
  // argv: groups of (T, r, n_kv, d); with --runs first: groups of (T, rk, rv, n_kv, d)
  if (argc > 1 && (std::string(argv[1]) == "--runs" || std::string(argv[1]) == "--runs-int8")) {
    const bool i8 = std::string(argv[1]) == "--runs-int8";
    int bad = 0, n = 0;
    for (int i = 2; i + 4 < argc; i += 5) {
      const int T = std::atoi(argv[i]), rk = std::atoi(argv[i + 1]), rv = std::atoi(argv[i + 2]),
                nkv = std::atoi(argv[i + 3]), d = std::atoi(argv[i + 4]);
      bad |= i8 ? check_runs_i8(T, rk, rv, nkv, d) : check_runs(T, rk, rv, nkv, d);
      ++n;
    }
    std::printf("%s (%d geometries)\n", bad ? "FAIL" : "OK", n);
    return bad;
  }
  int bad = 0, n = 0;
  for (int i = 1; i + 3 < argc; i += 4) {
    const int T = std::atoi(argv[i]), r = std::atoi(argv[i + 1]), nkv = std::atoi(argv[i + 2]),
              d = std::atoi(argv[i + 3]);
    for (int kind = 0; kind < 4; ++kind) bad |= check(kind, T, r, nkv, d);
    ++n;
  }
  std::printf("%s (%d geometries)\n", bad ? "FAIL" : "OK", n);
  return bad;
}
