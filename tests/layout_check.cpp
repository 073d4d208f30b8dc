// Host-only check of the packed fragment layout declared in milo_internal.h:
// for each geometry given on the command line, every element of the padded
// source block is produced by exactly one (fragment, lane, element) and every
// (fragment, lane, element) maps inside the padded block.
#include <cstdio>
#include <cstdlib>
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
  return 0;
}

int main(int argc, char** argv) {
  // argv: groups of (T, r, n_kv, d)
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
