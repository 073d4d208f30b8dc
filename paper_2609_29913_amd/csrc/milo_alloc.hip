// Device side of the entropy rank allocation (Sec. 4.3, Eqs. 5-7): a radix
// select of the k-th largest candidate singular value over all blocks, then
// per-block counts and the block-ordered hand-out of equal values.
#include <hip/hip_runtime.h>

#include <climits>

#include "milo_internal.h"

namespace milo {
namespace {

constexpr int kSelThreads = 256;
constexpr int kAssignThreads = 1024;

// The key of a singular value: its bit pattern without the sign bit (valid
// inputs are >= 0, so this only maps -0 to +0); non-negative floats order like
// their bit patterns.
__device__ inline uint32_t sv_key(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

__global__ __launch_bounds__(kSelThreads) void alloc_init_kernel(AllocState* st, uint32_t k) {
  st->hist[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    st->prefix = 0;
    st->mask = 0;
    st->k_rem = k;
    st->bad_block = INT_MAX;
  }
}

// One radix pass: histogram of digit (key >> shift) & 255 over the candidates
// whose higher bits match the prefix fixed so far.  One workgroup covers 256
// columns of one row; the first pass also checks every value of the row.
__global__ __launch_bounds__(kSelThreads) void alloc_hist_kernel(AllocArgs a, int shift, int check) {
  __shared__ uint32_t h[256];
  const int b = blockIdx.x / a.chunks;
  const int j = (blockIdx.x % a.chunks) * kSelThreads + threadIdx.x;
  h[threadIdx.x] = 0;
  __syncthreads();
  const AllocBounds bd = a.bounds[b];
  const uint32_t prefix = a.st->prefix, mask = a.st->mask;
  if (j < bd.n_sv) {
    const float* row = a.sigma + (int64_t)b * a.ld;
    const float x = row[j];
    if (check) {
      bool bad = !(x >= 0.0f) || !(x < __builtin_huge_valf());  // negative, infinite or NaN
      if (j + 1 < bd.n_sv && row[j + 1] > x) bad = true;         // increasing
      if (bad) atomicMin(&a.st->bad_block, b);
    }
    const uint32_t key = sv_key(x);
    if (j >= bd.lo && j < bd.hi && (key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
  }
  __syncthreads();
  const uint32_t v = h[threadIdx.x];
  if (v) atomicAdd(&a.st->hist[threadIdx.x], v);
}

// Picks the digit that holds the k_rem-th largest matching key, fixes it in
// the prefix and clears the histogram for the next pass.
__global__ __launch_bounds__(64) void alloc_pick_kernel(AllocState* st, int shift) {
  if (threadIdx.x == 0) {
    const uint32_t k = st->k_rem;
    uint32_t above = 0;
    int d = 255;
    for (; d > 0; --d) {
      const uint32_t c = st->hist[d];
      if (above + c >= k) break;
      above += c;
    }
    st->k_rem = k - above;
    st->prefix |= (uint32_t)d << shift;
    st->mask |= 255u << shift;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 256; i += 64) st->hist[i] = 0;
}

// Per block (one wave each): candidates above and equal to the selected key.
__global__ __launch_bounds__(kSelThreads) void alloc_count_kernel(AllocArgs a) {
  const int b = blockIdx.x * (kSelThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (b >= a.n_blocks) return;
  const AllocBounds bd = a.bounds[b];
  const uint32_t tau = a.st->prefix;
  const float* row = a.sigma + (int64_t)b * a.ld;
  int gt = 0, eq = 0;
  for (int j = bd.lo + lane; j < bd.hi; j += 64) {
    const uint32_t key = sv_key(row[j]);
    gt += key > tau ? 1 : 0;
    eq += key == tau ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    gt += __shfl_xor(gt, o);
    eq += __shfl_xor(eq, o);
  }
  if (lane == 0) {
    a.cnt[b] = gt;
    a.cnt[a.n_blocks + b] = eq;
  }
}

// One workgroup: an exclusive scan of the equal counts in block order; block b
// takes min(eq_b, remaining units) of the values equal to the selected key.
__global__ __launch_bounds__(kAssignThreads) void alloc_assign_kernel(AllocArgs a) {
  __shared__ int64_t wsum[kAssignThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t units = a.st->k_rem;
  int64_t carry = 0;
  for (int base = 0; base < a.n_blocks; base += kAssignThreads) {
    const int b = base + threadIdx.x;
    const int64_t eq = b < a.n_blocks ? a.cnt[a.n_blocks + b] : 0;
    int64_t x = eq;  // inclusive scan inside the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int64_t before = 0, total = 0;
    for (int w = 0; w < kAssignThreads / 64; ++w) {
      if (w < wave) before += wsum[w];
      total += wsum[w];
    }
    if (b < a.n_blocks) {
      const int64_t excl = carry + before + x - eq;
      int64_t take = units - excl;
      take = take < 0 ? 0 : (take > eq ? eq : take);
      a.ranks[b] = a.bounds[b].lo + a.cnt[b] + (int32_t)take;
    }
    carry += total;
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_allocate(const AllocArgs& a, uint32_t k, hipStream_t s, hipEvent_t* ev) {
  hipError_t e;
  if (ev && (e = hipEventRecord(ev[0], s)) != hipSuccess) return e;
  alloc_init_kernel<<<1, kSelThreads, 0, s>>>(a.st, k);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const unsigned grid = (unsigned)a.n_blocks * (unsigned)a.chunks;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (pass > 0 && k == 0) break;  // only the check
    if (ev && (e = hipEventRecord(ev[1 + 2 * pass], s)) != hipSuccess) return e;
    alloc_hist_kernel<<<grid, kSelThreads, 0, s>>>(a, shift, pass == 0 ? 1 : 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev && (e = hipEventRecord(ev[2 + 2 * pass], s)) != hipSuccess) return e;
    if (k == 0) break;
    alloc_pick_kernel<<<1, 64, 0, s>>>(a.st, shift);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (k > 0) {
    alloc_count_kernel<<<(a.n_blocks + 3) / 4, kSelThreads, 0, s>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    alloc_assign_kernel<<<1, kAssignThreads, 0, s>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (ev && (e = hipEventRecord(ev[9], s)) != hipSuccess) return e;
  return hipSuccess;
}

}  // namespace milo
