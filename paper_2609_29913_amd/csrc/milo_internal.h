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
// v_mfma_f32_32x32x16_bf16, so one wave loads one fragment with one fully
// coalesced 16-byte load per lane.  Rows beyond T_b and ranks beyond r are
// stored as zeros (token count padded to 32, ranks padded to 32).
//
// Lane l = 32*c + m (c = lane group 0/1, m = 0..31), element e = 0..7.
//   P^K frag (tau, kap):   P^K[32*tau + m][16*kap + 8*c + e]        (A: tokens x rank)
//   P^V frag (sig, rho):   P^V[16*sig + 8*c + e][32*rho + m]        (A: rank x tokens)
//   R^K frag (g, rho, kap): R^K[32*rho + m][g*d + 16*kap + 8*c + e] (A: rank x d)
//   R^V frag (g, dlt, kap): R^V[16*kap + 8*(e/4) + 4*c + e%4][g*d + 32*dlt + m]
//                                                                   (A: d x rank)
// The R^V rank order inside a 16-rank step matches the rows that one lane holds
// in the fp32 accumulator of a 32x32 MFMA (rows 8*(v/4) + 4*c + v%4), so the
// latent accumulator feeds the up-projection straight from registers.
// Fragment order: P^K [tau][kap], P^V [sig][rho], R^K [g][rho][kap], R^V [g][dlt][kap].
// ---------------------------------------------------------------------------
constexpr int kFragElems = 512;  // 64 lanes x 8 bf16
enum FactorKind : int { kPK = 0, kRK = 1, kPV = 2, kRV = 3 };

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
    default:  return (int64_t)f.n_kv * (f.d / 32) * (f.r_pad / 16);
  }
}

// Source (row, col) of element e of lane `lane` in fragment `frag`.
__host__ __device__ inline void frag_source(const FactorGeom& f, int64_t frag, int lane, int e,
                                            int* row, int* col) {
  const int m = lane & 31, c = lane >> 5;
  switch (f.kind) {
    case kPK: {
      const int nk = f.r_pad / 16;
      const int tau = (int)(frag / nk), kap = (int)(frag % nk);
      *row = 32 * tau + m;
      *col = 16 * kap + 8 * c + e;
      return;
    }
    case kPV: {
      const int nr = f.r_pad / 32;
      const int sig = (int)(frag / nr), rho = (int)(frag % nr);
      *row = 16 * sig + 8 * c + e;
      *col = 32 * rho + m;
      return;
    }
    case kRK: {
      const int nk = f.d / 16, nr = f.r_pad / 32;
      const int kap = (int)(frag % nk);
      const int rho = (int)((frag / nk) % nr);
      const int g = (int)(frag / ((int64_t)nk * nr));
      *row = 32 * rho + m;
      *col = g * f.d + 16 * kap + 8 * c + e;
      return;
    }
    default: {
      const int nk = f.r_pad / 16, nd = f.d / 32;
      const int kap = (int)(frag % nk);
      const int dlt = (int)((frag / nk) % nd);
      const int g = (int)(frag / ((int64_t)nk * nd));
      *row = 16 * kap + 8 * (e >> 2) + 4 * c + (e & 3);
      *col = g * f.d + 32 * dlt + m;
      return;
    }
  }
}

// Per-block metadata in device memory; offsets are in bf16 elements from the
// start of the cache's packed buffer.
struct BlockMeta {
  int64_t off_pk, off_rk, off_pv, off_rv;
  int32_t T, T_pad, rk_pad, rv_pad;
};

// Work item of the attention kernel (one workgroup each), as int4:
//   block task: {block id >= 0, partial slot, kv group g, column tile}
//   tail task:  {-1 - request i, partial slot, kv group g, tail chunk}
//   empty:      {kEmptyTask, 0, 0, 0}
constexpr int kEmptyTask = -0x7fffffff;

// Attention kernel geometry.
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kCols = 64;                      // query columns per workgroup
constexpr int kTokWave = 64;                   // tokens per wave per tile
constexpr int kTile = kWaves * kTokWave;       // tokens per tile
constexpr int kWStride = kTile + 8;            // bf16 row stride of the weight tile in LDS
constexpr int kORow = 68;                      // fp32 row stride of the up-projection reduction
constexpr int kMaxGroup = 16;                  // max query heads per KV head
constexpr int kMaxRank = 960;                  // largest supported rank (LDS bound)

struct AttendArgs {
  const uint16_t* data;      // packed factors
  const BlockMeta* meta;     // [n_blocks]
  const int4* tasks;         // [grid]
  const uint16_t* q;         // [n_q][H_q][d]
  const uint16_t* tail_k;    // [n_q][tail_cap][H_kv][d]
  const uint16_t* tail_v;
  const int32_t* tail_len;   // device [n_q]
  float* part_o;             // [n_q*H_q][n_slots][d]
  float2* part_ml;           // [n_q*H_q][n_slots] (max in log2 units, sum)
  float qscale;              // scale * log2(e)
  int n_q, H_q, H_kv, G;
  int tail_cap, tail_chunk;
  int n_slots;
  int qt_stride;             // bf16 row stride of the projected query in LDS
};

struct MergeArgs {
  const float* part_o;
  const float2* part_ml;
  const int32_t* tail_len;   // device [n_q]
  float* out;                // [n_q][H_q][d]
  int H_q, n_sel, n_slots, tail_chunk;
};

struct PackArgs {
  const uint16_t* src;
  uint16_t* dst;
  FactorGeom geom;
  int64_t n_frags;
};

// Launchers (defined in milo_kernels.hip).
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_attend(const AttendArgs& a, int head_dim, int max_rt, int grid, size_t lds_bytes,
                         hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, int head_dim, int n_cols, hipStream_t s);
size_t attend_lds_bytes(int head_dim, int rk_pad_max, int G, int tail_chunk);

}  // namespace milo
