// Encoder of the block-wise low-rank cache (Sec. 4.2 Eq. 3, Alg. 1 encoding
// stage): for every block K_b (T_b x D, bf16) its singular values and right
// singular vectors, then the truncated factors P = K_b V_r = U_r Sigma_r and
// R = V_r^T that milo_cache_create stores.  (The ranks r_b in between come
// from the entropy rank allocation, milo_allocate_ranks.)
//
//  gram_kernel     G_b = K_b^T K_b (bf16 MFMA, fp32 accumulation; D_pad x D_pad,
//                  zero-padded to a multiple of 64)
//  bj_*_kernel     the symmetric eigenproblem of G_b by block Jacobi: blocks of 32
//                  indices paired by the circle ordering; per round one launch
//                  sweeps every pair's 64 x 64 subproblem in LDS (scalar
//                  cyclic Jacobi), the next rotates the rest of G and V by the
//                  pair rotations (64 x 64 products in LDS); once per sweep the
//                  host learns whether any block still rotated.  Then the
//                  eigenvalues are sorted (bitonic, LDS), sigma = sqrt(max(lambda,
//                  0)), V^T written row by row
//  factor_kernel   P = K_b V_r (fp32 accumulation, bf16 out), R = V_r^T (bf16)
//
// Precision: the Gram matrix squares the condition number, so in fp32 the
// eigenvalues carry an absolute error of about 1e-7 .. 1e-6 lambda_max (more for
// flat spectra); singular values well below 1e-3 sigma_max are correspondingly
// less accurate.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <vector>

#include "milo.h"
#include "milo_internal.h"

namespace milo {
namespace {

constexpr int kMaxModel = 1024;      // largest D (= H_kv * d) the encoder handles
constexpr size_t kEncodeWorkspace = size_t(2) << 30;  // G, V and rotations of the blocks in flight
constexpr int kMaxEncodeBlocks = 65535;  // blocks per call (one grid z-slice or y-row each)
constexpr int kGramTile = 64;        // G tile per workgroup (four waves, a 32 x 32 quadrant each)
constexpr int kGramK = 32;           // tokens per LDS stage

__device__ __forceinline__ float bf(uint16_t u) { return __uint_as_float(static_cast<uint32_t>(u) << 16); }

// G_b[i][j] = sum_t K_b[t][i] K_b[t][j] over i, j < D; rows and columns
// D .. D_pad - 1 are zero.  One workgroup (four waves) per 64 x 64 tile of G:
// 32 tokens at a time go to LDS transposed ([dim][token], bf16) and each wave
// accumulates its 32 x 32 quadrant with v_mfma_f32_32x32x16_bf16 (products of
// bf16 values are exact in fp32; only the fp32 accumulation rounds).
// grid: (D_pad / 64)^2 x n_blocks.
typedef __bf16 bf16x8g __attribute__((ext_vector_type(8)));
typedef float f32x16g __attribute__((ext_vector_type(16)));
constexpr int kGramStride = kGramK + 8;  // bf16 row stride of a staged [dim][token] slice
__global__ __launch_bounds__(256) void gram_kernel(const uint16_t* const* k, const int32_t* tokens, int D, int Dp,
                                                   float* G_all) {
  __shared__ __align__(16) uint16_t a[kGramTile][kGramStride], c[kGramTile][kGramStride];
  const int b = blockIdx.z;
  const int T = tokens[b];
  const uint16_t* K = k[b];
  float* G = G_all + (size_t)b * Dp * Dp;
  const int tiles = Dp / kGramTile;
  const int i0 = (blockIdx.x % tiles) * kGramTile, j0 = (blockIdx.x / tiles) * kGramTile;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r0 = 32 * (w >> 1), c0 = 32 * (w & 1), m = lane & 31, hi = lane >> 5;
  f32x16g acc = {};
  for (int t0 = 0; t0 < T; t0 += kGramK) {
    // thread: token t0 + tid / 8, dims 8 (tid % 8) .. +7 of both tiles
    const int tt = tid >> 3, d8 = 8 * (tid & 7), t = t0 + tt;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int di = i0 + d8 + e, dj = j0 + d8 + e;
      a[d8 + e][tt] = (t < T && di < D) ? K[(int64_t)t * D + di] : (uint16_t)0;
      c[d8 + e][tt] = (t < T && dj < D) ? K[(int64_t)t * D + dj] : (uint16_t)0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGramK / 16; ++kk) {
      // A: G rows (dims of the i tile) x 16 tokens; B: 16 tokens x dims of the j tile
      const bf16x8g x = *reinterpret_cast<const bf16x8g*>(&a[r0 + m][16 * kk + 8 * hi]);
      const bf16x8g y = *reinterpret_cast<const bf16x8g*>(&c[c0 + m][16 * kk + 8 * hi]);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  // lane (hi, m) holds column c0 + m of rows r0 + 8 (i / 4) + 4 hi + i % 4
#pragma unroll
  for (int i = 0; i < 16; ++i) G[(size_t)(i0 + r0 + 8 * (i >> 2) + 4 * hi + (i & 3)) * Dp + j0 + c0 + m] = acc[i];
}

// Round `round` of the circle ordering of n (even) indices: pair t's members.
__device__ __forceinline__ void circle_pair(int n, int round, int t, int* p, int* q) {
  auto at = [&](int i) { return i == 0 ? 0 : 1 + (i - 1 + round) % (n - 1); };
  int x = at(t), y = at(n - 1 - t);
  *p = x < y ? x : y;
  *q = x < y ? y : x;
}

// Block Jacobi.  The D_pad indices form n_blk = D_pad / 32 blocks of 32; a
// sweep is n_blk - 1 rounds of the circle ordering over blocks, each round
// n_blk / 2 disjoint block pairs.  Pair (u, w)'s subproblem is the 64 x 64
// principal submatrix of G on blocks u and w: bj_solve_kernel rotates it by one
// cyclic Jacobi sweep in LDS (same threshold as the whole problem) and stores
// its rotation J; bj_apply_*_kernel then rotate the rest of G (G_pq <- J_p^T
// G_pq J_q between pairs) and V (V[:, pair p] <- V[:, pair p] J_p).  A sweep in
// which no subproblem needed a rotation leaves every off-diagonal entry of G
// below the threshold.
struct BJArgs {
  float* G;           // [n][D_pad][D_pad] row-major, symmetric
  float* V;           // [n][D_pad][D_pad], V[i][j] = component i of eigenvector j
  float* J;           // [n][n_pair][64][64] the round's pair rotations
  int* rot_pair;      // [n][n_pair] 1 if pair p's J is not the identity this round
  int* rot_mat;       // [n] 1 if any pair of the matrix rotated this sweep
  int* active;        // [n] 0 once a whole sweep found nothing to rotate
  float* floor_abs;   // [n] 1e-10 trace(G_b)
  unsigned* gemms;    // [n] 64^3 products executed (solves' re-orthogonalisation and applies)
  int Dp, n_blk, round;
  float tol;
};
constexpr int kBJ = 64;       // subproblem order (two blocks of 32)
constexpr int kBJS = kBJ + 1;  // LDS row stride
constexpr int kBJThreads = 256;    // init and apply kernels (the 64 x 64 products: one 32 x 32 quadrant per wave)
constexpr int kSolveThreads = 1024;  // subproblem sweep: one 2 x 2 block and two row pairs of J per thread per round
constexpr int kMaxSweeps = 30;

// V_b = I, floor_abs[b] = 1e-10 trace(G_b), the per-matrix flags cleared; grid: n.
__global__ __launch_bounds__(kBJThreads) void bj_init_kernel(BJArgs a, int* sweeps_used) {
  __shared__ float part[kBJThreads];
  const int b = blockIdx.x, tid = threadIdx.x, Dp = a.Dp;
  const float* G = a.G + (size_t)b * Dp * Dp;
  float* V = a.V + (size_t)b * Dp * Dp;
  for (int x = tid; x < Dp * Dp; x += kBJThreads) V[x] = (x / Dp == x % Dp) ? 1.f : 0.f;
  float tr = 0.f;
  for (int i = tid; i < Dp; i += kBJThreads) tr += G[(size_t)i * Dp + i];
  part[tid] = tr;
  __syncthreads();
  for (int w = kBJThreads / 2; w > 0; w /= 2) {
    if (tid < w) part[tid] += part[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    a.floor_abs[b] = 1e-10f * part[0];
    a.active[b] = 1;
    a.rot_mat[b] = 0;
    a.gemms[b] = 0;
    sweeps_used[b] = 0;
  }
}

// 64 x 64 x 64 products in LDS on four waves, by v_mfma_f32_32x32x2_f32: wave w
// of the four computes the 32 x 32 quadrant (rows 32 (w >> 1), columns
// 32 (w & 1)) of X^T Y (transpose_x) or X Y.  Operand lanes: A (row l % 32,
// k l / 32), B (k l / 32, column l % 32); the result in the 32 x 32 MFMA layout,
// lane l holding column l % 32 of rows 8 (i / 4) + 4 (l / 32) + i % 4, i = 0..15
// (bj_row, bj_col give its place in the 64 x 64 result).
typedef float f32x16e __attribute__((ext_vector_type(16)));
template <bool TRANSPOSE_X>
__device__ __forceinline__ f32x16e bj_product(const float (*X)[kBJS], const float (*Y)[kBJS]) {
  const int lane = threadIdx.x & 63, w = (threadIdx.x >> 6) & 3;
  const int r0 = 32 * (w >> 1), c0 = 32 * (w & 1), m = lane & 31, kk = lane >> 5;
  f32x16e acc = {};
#pragma unroll 8
  for (int k0 = 0; k0 < kBJ; k0 += 2) {
    const float x = TRANSPOSE_X ? X[k0 + kk][r0 + m] : X[r0 + m][k0 + kk];
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x, Y[k0 + kk][c0 + m], acc, 0, 0, 0);
  }
  return acc;
}
__device__ __forceinline__ int bj_row(int i) {
  return 32 * (((threadIdx.x >> 6) & 3) >> 1) + 8 * (i >> 2) + 4 * ((threadIdx.x & 63) >> 5) + (i & 3);
}
__device__ __forceinline__ int bj_col() { return 32 * ((threadIdx.x >> 6) & 1) + (threadIdx.x & 31); }

// Round rr of the circle ordering of the 64 subproblem indices, pair t (no division).
__device__ __forceinline__ void circle_pair64(int rr, int t, int* p, int* q) {
  auto at = [&](int i) {
    int x = i - 1 + rr;
    x = x >= kBJ - 1 ? x - (kBJ - 1) : x;
    return i == 0 ? 0 : 1 + x;
  };
  const int x = at(t), y = at(kBJ - 1 - t);
  *p = x < y ? x : y;
  *q = x < y ? y : x;
}

// One workgroup per (pair, matrix): one cyclic Jacobi sweep (63 rounds of 32
// disjoint rotations) over the pair's 64 x 64 subproblem in LDS.  (Solving the
// subproblem to convergence on every visit costs several sweeps per visit and
// saves at most one outer sweep, so each visit does one.)  As in Rutishauser's
// formulation, a rotated index pair's off-diagonal entry is set to zero and its
// diagonal entries become G_pp - t G_pq and G_qq + t G_pq (t = tan of the
// angle): this keeps the eigenvalues at the accuracy of the Gram matrix and lets
// rank-deficient blocks (T_b < D) converge.  The rotated subproblem goes back
// into G; J, made orthogonal to rounding by one Newton-Schulz step
// J (3 I - J^T J) / 2, goes to the rotation buffer for the apply kernels.
// grid: (n_blk / 2, n).
__global__ __launch_bounds__(kSolveThreads) void bj_solve_kernel(BJArgs a) {
  __shared__ float S[kBJ][kBJS], Jm[kBJ][kBJS], M[kBJ][kBJS];
  __shared__ float2 rot[kBJ / 2];  // (c, s) of index pair k this round
  __shared__ int pq[kBJ / 2];      // p | q << 8
  __shared__ float2 diag[kBJ / 2];  // (G_pp - t G_pq, G_qq + t G_pq) of a rotated pair
  __shared__ int any_rot;
  const int b = blockIdx.y, pair = blockIdx.x, tid = threadIdx.x, Dp = a.Dp;
  const int n_pair = a.n_blk / 2;
  if (!a.active[b]) return;
  int u, w;
  circle_pair(a.n_blk, a.round, pair, &u, &w);
  auto gi = [&](int i) { return i < 32 ? u * 32 + i : w * 32 + (i - 32); };
  float* G = a.G + (size_t)b * Dp * Dp;
  for (int x = tid; x < kBJ * kBJ; x += kSolveThreads) {
    const int i = x / kBJ, j = x % kBJ;
    S[i][j] = G[(size_t)gi(i) * Dp + gi(j)];
    Jm[i][j] = i == j ? 1.f : 0.f;
  }
  if (tid == 0) any_rot = 0;
  const float tol = a.tol, flo = a.floor_abs[b];
  // the 2 x 2 blocks (index pair k's rows, pair l's columns) with k <= l: 528 of
  // them, enumerated as 16 row pairs (k, 31 - k) of 33 blocks each
  constexpr int kHalf = kBJ / 2, kUpper = kHalf * (kHalf + 1) / 2;
  __syncthreads();
  for (int rr = 0; rr < kBJ - 1; ++rr) {
    if (tid < kHalf) {
      int p, q;
      circle_pair64(rr, tid, &p, &q);
      const float gpp = S[p][p], gqq = S[q][q], gpq = S[p][q];
      float c = 1.f, s = 0.f, tt = 0.f;
      if (gpq != 0.f && fabsf(gpq) > tol * sqrtf(fabsf(gpp) * fabsf(gqq)) && fabsf(gpq) > flo) {
        const float theta = (gqq - gpp) / (2.f * gpq);
        // t = sign(theta) / (|theta| + sqrt(1 + theta^2)); 1 / (2 theta) where theta^2 would overflow
        tt = fabsf(theta) > 1e18f ? 0.5f / theta
                                  : copysignf(1.f, theta) / (fabsf(theta) + sqrtf(1.f + theta * theta));
        c = 1.f / sqrtf(1.f + tt * tt);
        s = tt * c;
        any_rot = 1;  // benign race: every writer stores 1
      }
      rot[tid] = make_float2(c, s);
      pq[tid] = p | q << 8;
      diag[tid] = make_float2(gpp - tt * gpq, gqq + tt * gpq);
    }
    __syncthreads();
    // S <- R^T S R, one 2 x 2 block per item, the mirror block written as its transpose
#pragma unroll
    for (int m = 0; m < (kUpper + kSolveThreads - 1) / kSolveThreads; ++m) {
      const int x = tid + m * kSolveThreads;
      if (x >= kUpper) break;
      const int r = x / (kHalf + 1), c0 = x % (kHalf + 1);
      const bool first = c0 < kHalf - r;
      const int k = first ? r : kHalf - 1 - r;
      const int l = first ? r + c0 : k + (c0 - (kHalf - r));
      const float2 rk = rot[k], rl = rot[l];
      const float sk = rk.y, sl = rl.y;
      if (sk == 0.f && sl == 0.f) continue;
      const int pqk = pq[k];
      const int pk = pqk & 255, qk = pqk >> 8;
      if (k == l) {
        const float2 dg = diag[k];
        S[pk][qk] = 0.f;
        S[qk][pk] = 0.f;
        S[pk][pk] = dg.x;
        S[qk][qk] = dg.y;
        continue;
      }
      const int pql = pq[l];
      const int pl = pql & 255, ql = pql >> 8;
      const float ck = rk.x, cl = rl.x;
      const float e00 = S[pk][pl], e01 = S[pk][ql], e10 = S[qk][pl], e11 = S[qk][ql];
      // rows: r_p <- c r_p - s r_q, r_q <- s r_p + c r_q; then the same on columns
      const float f00 = ck * e00 - sk * e10, f01 = ck * e01 - sk * e11;
      const float f10 = sk * e00 + ck * e10, f11 = sk * e01 + ck * e11;
      const float g00 = cl * f00 - sl * f01, g01 = sl * f00 + cl * f01;
      const float g10 = cl * f10 - sl * f11, g11 = sl * f10 + cl * f11;
      S[pk][pl] = g00;
      S[pk][ql] = g01;
      S[qk][pl] = g10;
      S[qk][ql] = g11;
      S[pl][pk] = g00;
      S[ql][pk] = g01;
      S[pl][qk] = g10;
      S[ql][qk] = g11;
    }
    // J <- J R (columns p, q of every row): lane i of wave v takes row i and the
    // index pairs v, v + 16; the pairs' parameters are read before any update
    {
      const int i = tid % kBJ, v0 = tid / kBJ;
      constexpr int kPer = kHalf / (kSolveThreads / kBJ);
      float2 rk[kPer];
      int pqk[kPer];
#pragma unroll
      for (int m = 0; m < kPer; ++m) {
        rk[m] = rot[v0 + m * (kSolveThreads / kBJ)];
        pqk[m] = pq[v0 + m * (kSolveThreads / kBJ)];
      }
#pragma unroll
      for (int m = 0; m < kPer; ++m) {
        const float c = rk[m].x, s = rk[m].y;
        if (s == 0.f) continue;
        const int p = pqk[m] & 255, q = pqk[m] >> 8;
        const float jp = Jm[i][p], jq = Jm[i][q];
        Jm[i][p] = c * jp - s * jq;
        Jm[i][q] = s * jp + c * jq;
      }
    }
    __syncthreads();
  }
  const bool rotated = any_rot != 0;
  if (tid == 0) a.rot_pair[(size_t)b * n_pair + pair] = rotated ? 1 : 0;
  if (!rotated) return;
  for (int x = tid; x < kBJ * kBJ; x += kSolveThreads) {
    const int i = x / kBJ, j = x % kBJ;
    G[(size_t)gi(i) * Dp + gi(j)] = S[i][j];
  }
  // Newton-Schulz: M = J^T J, then J (3 I - M) / 2 = 1.5 J - 0.5 J M (the
  // products on the first four waves)
  if (tid < kBJThreads) {
    const f32x16e t = bj_product<true>(Jm, Jm);
#pragma unroll
    for (int i = 0; i < 16; ++i) M[bj_row(i)][bj_col()] = t[i];
  }
  __syncthreads();
  if (tid < kBJThreads) {
    const f32x16e t = bj_product<false>(Jm, M);
    float* Jout = a.J + ((size_t)b * n_pair + pair) * kBJ * kBJ;
#pragma unroll
    for (int i = 0; i < 16; ++i) Jout[bj_row(i) * kBJ + bj_col()] = 1.5f * Jm[bj_row(i)][bj_col()] - 0.5f * t[i];
  }
  if (tid == 0) {
    a.rot_mat[b] = 1;
    atomicAdd(&a.gemms[b], 2u);
  }
}

// The rest of a round, in two launches.  bj_apply_g_kernel: one workgroup per
// (off-diagonal pair block p < q of G, matrix): G_pq <- J_p^T G_pq J_q and G_qp
// its transpose.  bj_apply_v_kernel: one workgroup per (pair p, 64-row chunk
// of V, matrix): V[chunk rows][pair p columns] <- that slice J_p (two LDS
// tiles, so four workgroups fit per CU).  An identity J (a pair with no
// rotation) is skipped.  Rows of a pair's index set are two runs of 32, so
// 4-float groups are contiguous and 16-byte aligned in G, V and J.
__global__ __launch_bounds__(kBJThreads) void bj_apply_g_kernel(BJArgs a) {
  __shared__ float A[kBJ][kBJS], Jp[kBJ][kBJS], Jq[kBJ][kBJS];
  const int b = blockIdx.y, tid = threadIdx.x, Dp = a.Dp, n_pair = a.n_blk / 2;
  if (!a.active[b]) return;
  int task = blockIdx.x;
  const int* rot = a.rot_pair + (size_t)b * n_pair;
  const float* Jb = a.J + (size_t)b * n_pair * kBJ * kBJ;
  int p = 0;
  while (task >= n_pair - 1 - p) {
    task -= n_pair - 1 - p;
    ++p;
  }
  const int q = p + 1 + task;
  const bool rp = rot[p] != 0, rq = rot[q] != 0;
  if (!rp && !rq) return;
  int up, wp, uq, wq;
  circle_pair(a.n_blk, a.round, p, &up, &wp);
  circle_pair(a.n_blk, a.round, q, &uq, &wq);
  auto gp = [&](int i) { return i < 32 ? up * 32 + i : wp * 32 + (i - 32); };
  auto gq = [&](int i) { return i < 32 ? uq * 32 + i : wq * 32 + (i - 32); };
  float* G = a.G + (size_t)b * Dp * Dp;
  for (int x = tid; x < kBJ * kBJ / 4; x += kBJThreads) {
    const int i = x / (kBJ / 4), j = 4 * (x % (kBJ / 4));
    const float4 g = *reinterpret_cast<const float4*>(G + (size_t)gp(i) * Dp + gq(j));
    A[i][j] = g.x, A[i][j + 1] = g.y, A[i][j + 2] = g.z, A[i][j + 3] = g.w;
    if (rp) {
      const float4 v = *reinterpret_cast<const float4*>(Jb + ((size_t)p * kBJ + i) * kBJ + j);
      Jp[i][j] = v.x, Jp[i][j + 1] = v.y, Jp[i][j + 2] = v.z, Jp[i][j + 3] = v.w;
    }
    if (rq) {
      const float4 v = *reinterpret_cast<const float4*>(Jb + ((size_t)q * kBJ + i) * kBJ + j);
      Jq[i][j] = v.x, Jq[i][j + 1] = v.y, Jq[i][j + 2] = v.z, Jq[i][j + 3] = v.w;
    }
  }
  __syncthreads();
  if (rp) {
    const f32x16e t = bj_product<true>(Jp, A);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) A[bj_row(i)][bj_col()] = t[i];
    __syncthreads();
  }
  if (rq) {
    const f32x16e t = bj_product<false>(A, Jq);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) A[bj_row(i)][bj_col()] = t[i];
    __syncthreads();
  }
  for (int x = tid; x < kBJ * kBJ / 4; x += kBJThreads) {
    const int i = x / (kBJ / 4), j = 4 * (x % (kBJ / 4));
    *reinterpret_cast<float4*>(G + (size_t)gp(i) * Dp + gq(j)) = make_float4(A[i][j], A[i][j + 1], A[i][j + 2], A[i][j + 3]);
    *reinterpret_cast<float4*>(G + (size_t)gq(i) * Dp + gp(j)) = make_float4(A[j][i], A[j + 1][i], A[j + 2][i], A[j + 3][i]);
  }
  if (tid == 0) atomicAdd(&a.gemms[b], (rp ? 1u : 0u) + (rq ? 1u : 0u));
}

__global__ __launch_bounds__(kBJThreads) void bj_apply_v_kernel(BJArgs a) {
  __shared__ float A[kBJ][kBJS], Jp[kBJ][kBJS];
  const int b = blockIdx.y, tid = threadIdx.x, Dp = a.Dp, n_pair = a.n_blk / 2;
  if (!a.active[b]) return;
  const int p = blockIdx.x % n_pair, chunk = blockIdx.x / n_pair;
  if (!a.rot_pair[(size_t)b * n_pair + p]) return;
  int up, wp;
  circle_pair(a.n_blk, a.round, p, &up, &wp);
  auto gp = [&](int i) { return i < 32 ? up * 32 + i : wp * 32 + (i - 32); };
  const float* J = a.J + ((size_t)b * n_pair + p) * kBJ * kBJ;
  float* V = a.V + (size_t)b * Dp * Dp + (size_t)chunk * kBJ * Dp;
  for (int x = tid; x < kBJ * kBJ / 4; x += kBJThreads) {
    const int i = x / (kBJ / 4), j = 4 * (x % (kBJ / 4));
    const float4 v = *reinterpret_cast<const float4*>(V + (size_t)i * Dp + gp(j));
    A[i][j] = v.x, A[i][j + 1] = v.y, A[i][j + 2] = v.z, A[i][j + 3] = v.w;
    const float4 r = *reinterpret_cast<const float4*>(J + (size_t)i * kBJ + j);
    Jp[i][j] = r.x, Jp[i][j + 1] = r.y, Jp[i][j + 2] = r.z, Jp[i][j + 3] = r.w;
  }
  __syncthreads();
  const f32x16e t = bj_product<false>(A, Jp);
#pragma unroll
  for (int i = 0; i < 16; ++i) V[(size_t)bj_row(i) * Dp + gp(bj_col())] = t[i];
  if (tid == 0) atomicAdd(&a.gemms[b], 1u);
}

// End of a sweep: a matrix with no rotation in it is done; the others count the
// sweep.  *remaining = matrices still active.  grid: 1.
__global__ __launch_bounds__(1024) void bj_sweep_end_kernel(BJArgs a, int n, int sweep, int* sweeps_used,
                                                            int* remaining) {
  __shared__ int count;
  if (threadIdx.x == 0) count = 0;
  __syncthreads();
  int mine = 0;
  for (int b = threadIdx.x; b < n; b += 1024) {
    if (a.active[b]) {
      if (a.rot_mat[b]) {
        sweeps_used[b] = sweep + 1;
        ++mine;
      } else {
        a.active[b] = 0;
      }
    }
    a.rot_mat[b] = 0;
  }
  if (mine) atomicAdd(&count, mine);
  __syncthreads();
  if (threadIdx.x == 0) *remaining = count;
}

// Eigenvalues in descending order (bitonic sort of (lambda, index) over a power
// of two of entries; padding entries sort last), sigma = sqrt(max(lambda, 0)),
// and V^T row by row; grid: n.
__global__ __launch_bounds__(1024) void bj_finish_kernel(const float* G_all, const float* V_all, int D, int Dp,
                                                         float* sigma, float* vt) {
  __shared__ float key[kMaxModel];
  __shared__ int idx[kMaxModel];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* G = G_all + (size_t)b * Dp * Dp;
  const float* V = V_all + (size_t)b * Dp * Dp;
  int n2 = 1;
  while (n2 < Dp) n2 *= 2;
  for (int x = tid; x < n2; x += 1024) {
    const float g = x < D ? G[(size_t)x * Dp + x] : -INFINITY;
    key[x] = g == g ? g : -INFINITY;  // NaN (non-finite input) ranks with the padding, after every index < D
    idx[x] = x;
  }
  __syncthreads();
  for (int size = 2; size <= n2; size *= 2)
    for (int stride = size / 2; stride > 0; stride /= 2) {
      for (int x = tid; x < n2; x += 1024) {
        const int y = x ^ stride;
        if (y > x) {
          const bool desc = (x & size) == 0;
          const float kx = key[x], ky = key[y];
          const bool swap = desc ? (kx < ky || (kx == ky && idx[x] > idx[y])) : (kx > ky || (kx == ky && idx[x] < idx[y]));
          if (swap) {
            key[x] = ky;
            key[y] = kx;
            const int t = idx[x];
            idx[x] = idx[y];
            idx[y] = t;
          }
        }
      }
      __syncthreads();
    }
  for (int j = tid; j < D; j += 1024) sigma[(size_t)b * D + j] = sqrtf(fmaxf(key[j], 0.f));
  for (int x = tid; x < D * D; x += 1024) {
    const int j = x / D, col = x % D;
    const int src = idx[j] < D ? idx[j] : 0;  // always true: ties break by index, padding sorts after
    vt[((size_t)b * D + j) * D + col] = V[(size_t)col * Dp + src];
  }
}

// P_b = K_b V_r (T_b x r_b, bf16) and R_b = V_r^T (r_b x D, bf16); grid: one
// workgroup per (64 x 64 tile of P, block), R written by the tiles of column 0.
__global__ __launch_bounds__(256) void factor_kernel(const uint16_t* const* k, const int32_t* tokens,
                                                     const int32_t* ranks, int D, const float* vt_all,
                                                     uint16_t* const* p_out, uint16_t* const* r_out, int max_tiles_t) {
  __shared__ float a[kGramK][kGramTile + 1], c[kGramK][kGramTile + 1];
  const int b = blockIdx.z;
  const int T = tokens[b], r = ranks[b];
  const uint16_t* K = k[b];
  const float* VT = vt_all + (size_t)b * D * D;
  const int tt0 = (blockIdx.x % max_tiles_t) * kGramTile, j0 = (blockIdx.x / max_tiles_t) * kGramTile;
  if (tt0 >= T || j0 >= r) return;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < D; k0 += kGramK) {
    for (int x = threadIdx.x; x < kGramK * kGramTile; x += 256) {
      const int kk = x % kGramK, row = x / kGramK;
      const int t = tt0 + row, j = j0 + row, kc = k0 + kk;
      a[kk][row] = (t < T && kc < D) ? bf(K[(int64_t)t * D + kc]) : 0.f;
      c[kk][row] = (j < r && kc < D) ? VT[(size_t)j * D + kc] : 0.f;
    }
    __syncthreads();
    for (int kk = 0; kk < kGramK; ++kk)
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[kk][ty + 16 * u], c[kk][tx + 16 * v], acc[u][v]);
    __syncthreads();
  }
  uint16_t* P = p_out[b];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = tt0 + ty + 16 * u, j = j0 + tx + 16 * v;
      if (t < T && j < r) {
        const __bf16 h = (__bf16)acc[u][v];
        P[(int64_t)t * r + j] = *reinterpret_cast<const uint16_t*>(&h);
      }
    }
  if (tt0 == 0) {
    uint16_t* R = r_out[b];
    for (int x = threadIdx.x; x < kGramTile * D; x += 256) {
      const int j = j0 + x / D, col = x % D;
      if (j < r) {
        const __bf16 h = (__bf16)VT[(size_t)j * D + col];
        R[(int64_t)j * D + col] = *reinterpret_cast<const uint16_t*>(&h);
      }
    }
  }
}

int enc_fail(int code, const char* fmt, long long a = 0, long long b = 0) {
  char buf[256];
  std::snprintf(buf, sizeof buf, fmt, a, b);
  return report_error(code, buf);
}

// device copy of a host table (freed by the caller)
template <typename T>
hipError_t upload(const T* host, size_t n, T** dev, hipStream_t s) {
  hipError_t e = hipMalloc(reinterpret_cast<void**>(dev), n * sizeof(T));
  if (e != hipSuccess) return e;
  return hipMemcpyAsync(*dev, host, n * sizeof(T), hipMemcpyHostToDevice, s);
}

struct Encoding {
  int last_sweeps_max = 0;
  double last_flops = 0;
};
Encoding g_enc;

}  // namespace
}  // namespace milo

using namespace milo;

extern "C" int milo_block_svd(const uint16_t* const* k, const int32_t* tokens, int32_t n_blocks, int32_t d_model,
                              float* sigma, float* vt, void* hip_stream) {
  clear_error();
  if (!k || !tokens || !sigma || !vt) return enc_fail(MILO_ERR_INVALID_ARG, "NULL argument");
  if (n_blocks < 1 || n_blocks > kMaxEncodeBlocks)
    return enc_fail(MILO_ERR_INVALID_ARG, "n_blocks must be in [1, %lld] (got %lld)", kMaxEncodeBlocks, n_blocks);
  if (d_model < 1 || d_model > kMaxModel)
    return enc_fail(MILO_ERR_UNSUPPORTED, "d_model %lld outside [1, %lld]", d_model, kMaxModel);
  for (int b = 0; b < n_blocks; ++b) {
    if (!k[b]) return enc_fail(MILO_ERR_INVALID_ARG, "block %lld: NULL keys", b);
    if (tokens[b] < 1) return enc_fail(MILO_ERR_INVALID_ARG, "block %lld: T_b must be >= 1 (got %lld)", b, tokens[b]);
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  const int D = d_model, Dp = (D + kBJ - 1) / kBJ * kBJ;  // blocks of 32, an even number of them
  const int n_blk = Dp / 32, n_pair = n_blk / 2;
  // blocks in flight: their G, V and pair rotations within the workspace bound
  const size_t per_block = ((size_t)2 * Dp * Dp + (size_t)n_pair * kBJ * kBJ) * sizeof(float);
  const int chunk = (int)std::max<size_t>(1, std::min<size_t>(n_blocks, kEncodeWorkspace / per_block));
  const uint16_t** k_d = nullptr;
  int32_t* t_d = nullptr;
  float *G = nullptr, *V = nullptr, *J = nullptr;
  int* flags = nullptr;
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(s);
    (void)hipFree(k_d);
    (void)hipFree(t_d);
    (void)hipFree(G);
    (void)hipFree(V);
    (void)hipFree(J);
    (void)hipFree(flags);
  };
  auto hfail = [&](hipError_t e, const char* what) {
    cleanup();
    char buf[256];
    std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
    return report_error(e == hipErrorOutOfMemory ? MILO_ERR_OUT_OF_MEMORY : MILO_ERR_HIP, buf);
  };
  hipError_t e;
  if ((e = upload(k, n_blocks, const_cast<const uint16_t***>(&k_d), s)) != hipSuccess) return hfail(e, "key table");
  if ((e = upload(tokens, n_blocks, &t_d, s)) != hipSuccess) return hfail(e, "token counts");
  const size_t mat = (size_t)chunk * Dp * Dp;
  if ((e = hipMalloc(&G, mat * sizeof(float))) != hipSuccess) return hfail(e, "Gram workspace");
  if ((e = hipMalloc(&V, mat * sizeof(float))) != hipSuccess) return hfail(e, "eigenvector workspace");
  if ((e = hipMalloc(&J, (size_t)chunk * n_pair * kBJ * kBJ * sizeof(float))) != hipSuccess)
    return hfail(e, "rotation workspace");
  // per block: rot_pair [n_pair], rot_mat, active, floor_abs, gemms, sweeps_used; then `remaining`
  const size_t n_flags = (size_t)chunk * (n_pair + 5) + 1;
  if ((e = hipMalloc(&flags, n_flags * sizeof(int))) != hipSuccess) return hfail(e, "sweep flags");
  BJArgs a{};
  a.G = G;
  a.V = V;
  a.J = J;
  a.rot_pair = flags;
  a.rot_mat = a.rot_pair + (size_t)chunk * n_pair;
  a.active = a.rot_mat + chunk;
  a.floor_abs = reinterpret_cast<float*>(a.active + chunk);
  a.gemms = reinterpret_cast<unsigned*>(a.floor_abs + chunk);
  int* sweeps_d = reinterpret_cast<int*>(a.gemms + chunk);
  int* remaining_d = sweeps_d + chunk;
  a.Dp = Dp;
  a.n_blk = n_blk;
  a.tol = 1e-6f;
  const int tiles = Dp / kGramTile;
  int sweeps_max = 0;
  double flops = 0;
  std::vector<int> sw(chunk);
  std::vector<unsigned> gm(chunk);
  for (int b0 = 0; b0 < n_blocks; b0 += chunk) {
    const int nb = std::min(chunk, n_blocks - b0);
    hipLaunchKernelGGL(gram_kernel, dim3(tiles * tiles, 1, nb), dim3(256), 0, s, k_d + b0, t_d + b0, D, Dp, G);
    if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "gram kernel");
    hipLaunchKernelGGL(bj_init_kernel, dim3(nb), dim3(kBJThreads), 0, s, a, sweeps_d);
    if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "jacobi init kernel");
    for (int sweep = 0; sweep < kMaxSweeps; ++sweep) {
      for (int round = 0; round < n_blk - 1; ++round) {
        a.round = round;
        hipLaunchKernelGGL(bj_solve_kernel, dim3(n_pair, nb), dim3(kSolveThreads), 0, s, a);
        if (n_pair > 1)
          hipLaunchKernelGGL(bj_apply_g_kernel, dim3(n_pair * (n_pair - 1) / 2, nb), dim3(kBJThreads), 0, s, a);
        hipLaunchKernelGGL(bj_apply_v_kernel, dim3(n_pair * (Dp / kBJ), nb), dim3(kBJThreads), 0, s, a);
      }
      hipLaunchKernelGGL(bj_sweep_end_kernel, dim3(1), dim3(1024), 0, s, a, nb, sweep, sweeps_d, remaining_d);
      if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "jacobi kernels");
      int remaining = 0;
      if ((e = hipMemcpyAsync(&remaining, remaining_d, sizeof(int), hipMemcpyDeviceToHost, s)) != hipSuccess)
        return hfail(e, "active block count");
      if ((e = hipStreamSynchronize(s)) != hipSuccess) return hfail(e, "hipStreamSynchronize");
      if (remaining == 0) break;
    }
    hipLaunchKernelGGL(bj_finish_kernel, dim3(nb), dim3(1024), 0, s, G, V, D, Dp, sigma + (size_t)b0 * D,
                       vt + (size_t)b0 * D * D);
    if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "jacobi finish kernel");
    if ((e = hipMemcpyAsync(sw.data(), sweeps_d, nb * sizeof(int), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipMemcpyAsync(gm.data(), a.gemms, nb * sizeof(unsigned), hipMemcpyDeviceToHost, s)) != hipSuccess)
      return hfail(e, "sweep counts");
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return hfail(e, "hipStreamSynchronize");
    for (int i = 0; i < nb; ++i) {
      sweeps_max = std::max(sweeps_max, sw[i]);
      flops += 2.0 * kBJ * kBJ * kBJ * gm[i] + 2.0 * tokens[b0 + i] * (double)D * D;
    }
  }
  g_enc.last_sweeps_max = sweeps_max;
  g_enc.last_flops = flops;
  cleanup();
  return MILO_OK;
}

extern "C" int milo_block_svd_sweeps(int32_t* sweeps) {
  clear_error();
  if (!sweeps) return enc_fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *sweeps = g_enc.last_sweeps_max;
  return MILO_OK;
}

extern "C" int milo_block_svd_flops(double* flops) {
  clear_error();
  if (!flops) return enc_fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *flops = g_enc.last_flops;
  return MILO_OK;
}

extern "C" int milo_block_factors(const uint16_t* const* k, const int32_t* tokens, int32_t n_blocks, int32_t d_model,
                                  const float* vt, const int32_t* ranks, uint16_t* const* p_out, uint16_t* const* r_out,
                                  void* hip_stream) {
  clear_error();
  if (!k || !tokens || !vt || !ranks || !p_out || !r_out) return enc_fail(MILO_ERR_INVALID_ARG, "NULL argument");
  if (n_blocks < 1 || n_blocks > kMaxEncodeBlocks)
    return enc_fail(MILO_ERR_INVALID_ARG, "n_blocks must be in [1, %lld] (got %lld)", kMaxEncodeBlocks, n_blocks);
  if (d_model < 1 || d_model > kMaxModel)
    return enc_fail(MILO_ERR_UNSUPPORTED, "d_model %lld outside [1, %lld]", d_model, kMaxModel);
  int max_t = 0, max_r = 0;
  for (int b = 0; b < n_blocks; ++b) {
    if (!k[b] || !p_out[b] || !r_out[b]) return enc_fail(MILO_ERR_INVALID_ARG, "block %lld: NULL pointer", b);
    if (tokens[b] < 1) return enc_fail(MILO_ERR_INVALID_ARG, "block %lld: T_b must be >= 1 (got %lld)", b, tokens[b]);
    if (ranks[b] < 1 || ranks[b] > std::min(tokens[b], d_model))
      return enc_fail(MILO_ERR_INVALID_ARG, "block %lld: rank %lld outside [1, min(T_b, D)]", b, ranks[b]);
    max_t = std::max(max_t, (int)tokens[b]);
    max_r = std::max(max_r, (int)ranks[b]);
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  const uint16_t** k_d = nullptr;
  uint16_t **p_d = nullptr, **r_d = nullptr;
  int32_t *t_d = nullptr, *rk_d = nullptr;
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(s);
    (void)hipFree(k_d);
    (void)hipFree(p_d);
    (void)hipFree(r_d);
    (void)hipFree(t_d);
    (void)hipFree(rk_d);
  };
  auto hfail = [&](hipError_t e, const char* what) {
    cleanup();
    char buf[256];
    std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
    return report_error(e == hipErrorOutOfMemory ? MILO_ERR_OUT_OF_MEMORY : MILO_ERR_HIP, buf);
  };
  hipError_t e;
  if ((e = upload(k, n_blocks, const_cast<const uint16_t***>(&k_d), s)) != hipSuccess) return hfail(e, "key table");
  if ((e = upload(const_cast<uint16_t**>(p_out), n_blocks, &p_d, s)) != hipSuccess) return hfail(e, "P table");
  if ((e = upload(const_cast<uint16_t**>(r_out), n_blocks, &r_d, s)) != hipSuccess) return hfail(e, "R table");
  if ((e = upload(tokens, n_blocks, &t_d, s)) != hipSuccess) return hfail(e, "token counts");
  if ((e = upload(ranks, n_blocks, &rk_d, s)) != hipSuccess) return hfail(e, "ranks");
  const int tiles_t = (max_t + kGramTile - 1) / kGramTile, tiles_r = (max_r + kGramTile - 1) / kGramTile;
  hipLaunchKernelGGL(factor_kernel, dim3(tiles_t * tiles_r, 1, n_blocks), dim3(256), 0, s, k_d, t_d, rk_d, d_model, vt,
                     p_d, r_d, tiles_t);
  if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "factor kernel");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hfail(e, "hipStreamSynchronize");
  cleanup();
  return MILO_OK;
}
