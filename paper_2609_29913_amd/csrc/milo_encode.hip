// Encoder of the block-wise low-rank cache (Sec. 4.2 Eq. 3, Alg. 1 encoding
// stage): for every block K_b (T_b x D, bf16) its singular values and right
// singular vectors, then the truncated factors P = K_b V_r = U_r Sigma_r and
// R = V_r^T that milo_cache_create stores.  (The ranks r_b in between come
// from the entropy rank allocation, milo_allocate_ranks.)
//
//  gram_kernel     G_b = K_b^T K_b (fp32, D_pad x D_pad, zero-padded to an even size)
//  jacobi_kernel   one workgroup per block: the symmetric eigenproblem of G_b by
//                  parallel cyclic Jacobi (circle ordering: D_pad / 2 disjoint
//                  rotations per round, D_pad - 1 rounds per sweep), rotations
//                  accumulated into V; eigenvalues sorted (bitonic, LDS), sigma =
//                  sqrt(max(lambda, 0)), V^T written row by row
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
constexpr int kJacobiThreads = 1024;
constexpr int kMaxEncodeBlocks = 65535;  // blocks per call (one grid z-slice or workgroup each)
constexpr int kGramTile = 64;        // G tile per workgroup (256 threads, 4 x 4 outputs each)
constexpr int kGramK = 32;           // tokens per LDS stage

__device__ __forceinline__ float bf(uint16_t u) { return __uint_as_float(static_cast<uint32_t>(u) << 16); }

// G_b[i][j] = sum_t K_b[t][i] K_b[t][j] over i, j < D (tokens in order); rows and
// columns D .. D_pad - 1 are zero.  grid: (D_pad / 64 rounded up)^2 x n_blocks.
__global__ __launch_bounds__(256) void gram_kernel(const uint16_t* const* k, const int32_t* tokens, int D, int Dp,
                                                   float* G_all) {
  __shared__ float a[kGramK][kGramTile + 1], c[kGramK][kGramTile + 1];
  const int b = blockIdx.z;
  const int T = tokens[b];
  const uint16_t* K = k[b];
  float* G = G_all + (size_t)b * Dp * Dp;
  const int tiles = (Dp + kGramTile - 1) / kGramTile;
  const int i0 = (blockIdx.x % tiles) * kGramTile, j0 = (blockIdx.x / tiles) * kGramTile;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  for (int t0 = 0; t0 < T; t0 += kGramK) {
    for (int x = threadIdx.x; x < kGramK * kGramTile; x += 256) {
      const int tt = x / kGramTile, col = x % kGramTile, t = t0 + tt;
      a[tt][col] = (t < T && i0 + col < D) ? bf(K[(int64_t)t * D + i0 + col]) : 0.f;
      c[tt][col] = (t < T && j0 + col < D) ? bf(K[(int64_t)t * D + j0 + col]) : 0.f;
    }
    __syncthreads();
    for (int tt = 0; tt < kGramK; ++tt)
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[tt][ty + 16 * u], c[tt][tx + 16 * v], acc[u][v]);
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = i0 + ty + 16 * u, j = j0 + tx + 16 * v;
      if (i < Dp && j < Dp) G[(size_t)i * Dp + j] = acc[u][v];
    }
}

// Round `round` of the circle ordering of n (even) indices: pair t's members.
__device__ __forceinline__ void circle_pair(int n, int round, int t, int* p, int* q) {
  auto at = [&](int i) { return i == 0 ? 0 : 1 + (i - 1 + round) % (n - 1); };
  int x = at(t), y = at(n - 1 - t);
  *p = x < y ? x : y;
  *q = x < y ? y : x;
}

// One workgroup per block: cyclic Jacobi on G_b (in place, global memory),
// V_b accumulating the rotations, until a whole sweep finds no pair with
// |G_pq| > tol sqrt(|G_pp G_qq|) and |G_pq| > 1e-10 trace(G) (or max_sweeps);
// then sigma and V^T.  As in Rutishauser's formulation, a rotated pair's
// off-diagonal entry is set to zero and its diagonal entries are updated as
// G_pp - t G_pq and G_qq + t G_pq (t = tan of the angle) rather than taken from
// the rotated rows: this keeps the eigenvalues at the accuracy of the Gram
// matrix and lets rank-deficient blocks (T_b < D) converge.
__global__ __launch_bounds__(kJacobiThreads) void jacobi_kernel(float* G_all, float* V_all, int D, int Dp, float tol,
                                                                int max_sweeps, float* sigma, float* vt,
                                                                int* sweeps_used) {
  __shared__ float cs[kMaxModel / 2], sn[kMaxModel / 2], tn[kMaxModel / 2];
  __shared__ float dp[kMaxModel / 2], dq[kMaxModel / 2], od[kMaxModel / 2];
  __shared__ int pp[kMaxModel / 2], qq[kMaxModel / 2];
  __shared__ float floor_abs;
  __shared__ float key[kMaxModel];
  __shared__ int idx[kMaxModel];
  __shared__ int any_rot;
  const int b = blockIdx.x, tid = threadIdx.x;
  float* G = G_all + (size_t)b * Dp * Dp;
  float* V = V_all + (size_t)b * Dp * Dp;
  const int half = Dp / 2;
  for (int x = tid; x < Dp * Dp; x += kJacobiThreads) V[x] = (x / Dp == x % Dp) ? 1.f : 0.f;
  if (tid == 0) {
    float tr = 0.f;
    for (int i = 0; i < Dp; ++i) tr += G[(size_t)i * Dp + i];
    floor_abs = 1e-10f * tr;
  }
  __syncthreads();
  int sweep = 0;
  for (; sweep < max_sweeps; ++sweep) {
    if (tid == 0) any_rot = 0;
    __syncthreads();
    for (int round = 0; round < Dp - 1; ++round) {
      // rotation of each pair (classical Jacobi: annihilates G_pq)
      for (int t = tid; t < half; t += kJacobiThreads) {
        int p, q;
        circle_pair(Dp, round, t, &p, &q);
        const float gpp = G[(size_t)p * Dp + p], gqq = G[(size_t)q * Dp + q], gpq = G[(size_t)p * Dp + q];
        float c = 1.f, s = 0.f, tt = 0.f;
        if (gpq != 0.f && fabsf(gpq) > tol * sqrtf(fabsf(gpp) * fabsf(gqq)) && fabsf(gpq) > floor_abs) {
          const float theta = (gqq - gpp) / (2.f * gpq);
          // t = sign(theta) / (|theta| + sqrt(1 + theta^2)); 1 / (2 theta) where theta^2 would overflow
          tt = fabsf(theta) > 1e18f ? 0.5f / theta
                                    : copysignf(1.f, theta) / (fabsf(theta) + sqrtf(1.f + theta * theta));
          c = 1.f / sqrtf(1.f + tt * tt);
          s = tt * c;
          any_rot = 1;  // benign race: every writer stores 1
        }
        pp[t] = p;
        qq[t] = q;
        cs[t] = c;
        sn[t] = s;
        tn[t] = tt;
        dp[t] = gpp;
        dq[t] = gqq;
        od[t] = gpq;
      }
      __syncthreads();
      // rows p, q: G <- J^T G
      for (int x = tid; x < half * Dp; x += kJacobiThreads) {
        const int t = x / Dp, j = x % Dp;
        const float c = cs[t], s = sn[t];
        if (s == 0.f) continue;
        float* rp = G + (size_t)pp[t] * Dp + j;
        float* rq = G + (size_t)qq[t] * Dp + j;
        const float gp = *rp, gq = *rq;
        *rp = c * gp - s * gq;
        *rq = s * gp + c * gq;
      }
      __syncthreads();
      // columns p, q: G <- G J, V <- V J
      for (int x = tid; x < Dp * half; x += kJacobiThreads) {
        const int i = x / half, t = x % half;
        const float c = cs[t], s = sn[t];
        if (s == 0.f) continue;
        const int p = pp[t], q = qq[t];
        float* g = G + (size_t)i * Dp;
        const float gp = g[p], gq = g[q];
        g[p] = c * gp - s * gq;
        g[q] = s * gp + c * gq;
        float* v = V + (size_t)i * Dp;
        const float vp = v[p], vq = v[q];
        v[p] = c * vp - s * vq;
        v[q] = s * vp + c * vq;
      }
      __syncthreads();
      // the rotated 2 x 2 blocks, exactly diagonal
      for (int t = tid; t < half; t += kJacobiThreads) {
        if (sn[t] == 0.f) continue;
        const int p = pp[t], q = qq[t];
        G[(size_t)p * Dp + q] = 0.f;
        G[(size_t)q * Dp + p] = 0.f;
        G[(size_t)p * Dp + p] = dp[t] - tn[t] * od[t];
        G[(size_t)q * Dp + q] = dq[t] + tn[t] * od[t];
      }
      __syncthreads();
    }
    const bool done = any_rot == 0;
    __syncthreads();
    if (done) break;
  }
  // eigenvalues in descending order (bitonic sort of (lambda, index) over a
  // power of two of entries; padding entries sort last)
  int n2 = 1;
  while (n2 < Dp) n2 *= 2;
  for (int x = tid; x < n2; x += kJacobiThreads) {
    const float g = x < D ? G[(size_t)x * Dp + x] : -INFINITY;
    key[x] = g == g ? g : -INFINITY;  // NaN (non-finite input) ranks with the padding, after every index < D
    idx[x] = x;
  }
  __syncthreads();
  for (int size = 2; size <= n2; size *= 2)
    for (int stride = size / 2; stride > 0; stride /= 2) {
      for (int x = tid; x < n2; x += kJacobiThreads) {
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
  for (int j = tid; j < D; j += kJacobiThreads) sigma[(size_t)b * D + j] = sqrtf(fmaxf(key[j], 0.f));
  for (int x = tid; x < D * D; x += kJacobiThreads) {
    const int j = x / D, col = x % D;
    const int src = idx[j] < D ? idx[j] : 0;  // always true: ties break by index, padding sorts after
    vt[((size_t)b * D + j) * D + col] = V[(size_t)col * Dp + src];
  }
  if (tid == 0) sweeps_used[b] = sweep;
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
  const int D = d_model, Dp = D + (D & 1);
  const uint16_t** k_d = nullptr;
  int32_t* t_d = nullptr;
  float *G = nullptr, *V = nullptr;
  int* sw_d = nullptr;
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(s);
    (void)hipFree(k_d);
    (void)hipFree(t_d);
    (void)hipFree(G);
    (void)hipFree(V);
    (void)hipFree(sw_d);
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
  const size_t mat = (size_t)n_blocks * Dp * Dp;
  if ((e = hipMalloc(&G, mat * sizeof(float))) != hipSuccess) return hfail(e, "Gram workspace");
  if ((e = hipMalloc(&V, mat * sizeof(float))) != hipSuccess) return hfail(e, "eigenvector workspace");
  if ((e = hipMalloc(&sw_d, n_blocks * sizeof(int))) != hipSuccess) return hfail(e, "sweep counts");
  const int tiles = (Dp + kGramTile - 1) / kGramTile;
  hipLaunchKernelGGL(gram_kernel, dim3(tiles * tiles, 1, n_blocks), dim3(256), 0, s, k_d, t_d, D, Dp, G);
  if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "gram kernel");
  hipLaunchKernelGGL(jacobi_kernel, dim3(n_blocks), dim3(kJacobiThreads), 0, s, G, V, D, Dp, 1e-6f, 30, sigma, vt,
                     sw_d);
  if ((e = hipGetLastError()) != hipSuccess) return hfail(e, "jacobi kernel");
  std::vector<int> sw(n_blocks);
  if ((e = hipMemcpyAsync(sw.data(), sw_d, n_blocks * sizeof(int), hipMemcpyDeviceToHost, s)) != hipSuccess)
    return hfail(e, "sweep counts");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hfail(e, "hipStreamSynchronize");
  g_enc.last_sweeps_max = *std::max_element(sw.begin(), sw.end());
  cleanup();
  return MILO_OK;
}

extern "C" int milo_block_svd_sweeps(int32_t* sweeps) {
  clear_error();
  if (!sweeps) return enc_fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *sweeps = g_enc.last_sweeps_max;
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
