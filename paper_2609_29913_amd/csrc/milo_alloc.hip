// Device side of the entropy rank allocation (Sec. 4.3, Eqs. 5-7): a radix
// select of the k-th largest candidate singular value over all blocks (four
// histogram passes of 8 bits), then per-block counts and the block-ordered
// hand-out of equal values.
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

constexpr int kHistGrid = 1024;  // histogram workgroups at most (grid-stride over row chunks)

__global__ __launch_bounds__(kSelThreads) void alloc_init_kernel(AllocState* st, uint32_t k) {
#pragma unroll
  for (int p = 0; p < 4; ++p) st->hist[p][threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    st->k = k;
    st->bad_block = INT_MAX;
  }
}

// The digits picked by the first `passes` radix passes, derived by one wave
// (every lane gets the result): in pass p, the digit is the one whose bin holds
// the k_rem-th largest key among those matching the prefix fixed so far; k_rem
// then drops by the keys in higher bins.  Lane l holds bins 4l .. 4l+3.
__device__ inline void replay_picks(const AllocState* st, int passes, uint32_t& prefix, uint32_t& mask,
                                    uint32_t& k_rem) {
  const int lane = threadIdx.x & 63;
  uint32_t k = st->k;
  prefix = 0;
  mask = 0;
  uint4 hp[4];  // every pass's bins first: the loads do not depend on the picks
#pragma unroll
  for (int p = 0; p < 4; ++p)
    if (p < passes) hp[p] = *reinterpret_cast<const uint4*>(&st->hist[p][4 * lane]);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    if (p >= passes) break;
    const uint4 h = hp[p];
    const uint32_t own = h.x + h.y + h.z + h.w;
    uint32_t suf = own;  // keys in bins >= 4 * lane
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_down(suf, o);
      if (lane + o < 64) suf += y;
    }
    // suf does not increase with the lane and lane 0 holds every matching key
    // (>= k), so the lanes with suf >= k are 0 .. L
    const int L = __popcll(__ballot(suf >= k)) - 1;
    uint32_t above = __shfl(suf - own, L);
    const uint32_t b3 = __shfl(h.w, L), b2 = __shfl(h.z, L), b1 = __shfl(h.y, L);
    int d = 4 * L + 3;
    if (above + b3 < k) {
      above += b3;
      --d;
      if (above + b2 < k) {
        above += b2;
        --d;
        if (above + b1 < k) {
          above += b1;
          --d;
        }
      }
    }
    k -= above;
    prefix |= (uint32_t)d << (24 - 8 * p);
    mask |= 255u << (24 - 8 * p);
  }
  k_rem = k;
}

// Radix pass `pass`: histogram of digit (key >> (24 - 8 pass)) & 255 over the
// candidates whose higher bits match the digits picked so far.  A workgroup
// walks 256-column chunks of the rows; the first pass also checks every value.
__global__ __launch_bounds__(kSelThreads) void alloc_hist_kernel(AllocArgs a, int pass) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  uint32_t prefix, mask, k_rem;
  replay_picks(a.st, pass, prefix, mask, k_rem);
  __syncthreads();
  const int shift = 24 - 8 * pass;
  const int items = a.n_blocks * a.chunks;
  for (int it = blockIdx.x; it < items; it += gridDim.x) {
    const int b = it / a.chunks;
    const int j = (it % a.chunks) * kSelThreads + threadIdx.x;
    const AllocBounds bd = a.bounds[b];
    if (j < bd.n_sv) {
      const float* row = a.sigma + (int64_t)b * a.ld;
      const float x = row[j];
      if (pass == 0) {
        bool bad = !(x >= 0.0f) || !(x < __builtin_huge_valf());  // negative, infinite or NaN
        if (j + 1 < bd.n_sv && row[j + 1] > x) bad = true;         // increasing
        if (bad) atomicMin(&a.st->bad_block, b);
      }
      const uint32_t key = sv_key(x);
      if (j >= bd.lo && j < bd.hi && (key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
    }
  }
  __syncthreads();
  const uint32_t v = h[threadIdx.x];
  if (v) atomicAdd(&a.st->hist[pass][threadIdx.x], v);
}

// Per block (one wave each): candidates above and equal to the selected key.
__global__ __launch_bounds__(kSelThreads) void alloc_count_kernel(AllocArgs a) {
  const int b = blockIdx.x * (kSelThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (b >= a.n_blocks) return;
  const AllocBounds bd = a.bounds[b];
  uint32_t tau, mask, k_rem;
  replay_picks(a.st, 4, tau, mask, k_rem);
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
  uint32_t tau, mask, k_rem;
  replay_picks(a.st, 4, tau, mask, k_rem);
  const int64_t units = k_rem;
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
  const int items = a.n_blocks * a.chunks;
  const unsigned grid = (unsigned)(items < kHistGrid ? items : kHistGrid);
  for (int pass = 0; pass < (k == 0 ? 1 : 4); ++pass) {
    if (ev && (e = hipEventRecord(ev[1 + 2 * pass], s)) != hipSuccess) return e;
    alloc_hist_kernel<<<grid, kSelThreads, 0, s>>>(a, pass);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev && (e = hipEventRecord(ev[2 + 2 * pass], s)) != hipSuccess) return e;
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
