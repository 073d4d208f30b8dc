// Entropy rank allocation of the encoder (Sec. 4.3, Eqs. 5-7): the device side
// (a radix select of the k-th largest candidate singular value over all blocks
// in four histogram passes of 8 bits, then per-block counts and the
// block-ordered hand-out of equal values) and the host entry point
// milo_allocate_ranks of the C ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <vector>

#include "milo.h"
#include "milo_alloc.h"
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
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int c = 0; c < kHistCopies; ++c) st->hist[p][c][threadIdx.x] = 0;
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
  uint4 hp[4];  // every pass's bins (summed over the copies) first: the loads do not depend on the picks
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    hp[p] = make_uint4(0, 0, 0, 0);
    if (p < passes)
#pragma unroll
      for (int c = 0; c < kHistCopies; ++c) {
        const uint4 v = *reinterpret_cast<const uint4*>(&st->hist[p][c][4 * lane]);
        hp[p].x += v.x;
        hp[p].y += v.y;
        hp[p].z += v.z;
        hp[p].w += v.w;
      }
  }
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
// walks 256-column chunks of the rows and adds its LDS histogram into the copy
// of its XCD (almost every value shares the high digits, so one shared copy
// would put every workgroup's atomics on the same few bins); the first pass
// also checks every value.
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
  if (v) atomicAdd(&a.st->hist[pass][blockIdx.x % kHistCopies][threadIdx.x], v);
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

// ---------------------------------------------------------------------------
// Host entry point (C ABI, include/milo.h)
// ---------------------------------------------------------------------------
namespace {

using namespace milo;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return report_error(code, buf);
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

struct AllocTiming {  // measurement only: summed durations while timing is enabled
  std::mutex mu;
  double chain_ms = 0.0;  // whole kernel chain
  double hist_ms = 0.0;   // the histogram passes
  int64_t calls = 0;
};
AllocTiming g_alloc_timing;

}  // namespace

extern "C" {

int milo_allocate_ranks(const float* sigma, int64_t ld, int32_t n_blocks, const int32_t* n_sv, int64_t r_total,
                        int32_t r_min, int32_t r_max, int32_t* ranks, void* hip_stream) {
  clear_error();
  if (!sigma || !n_sv || !ranks) return fail(MILO_ERR_INVALID_ARG, "sigma, n_sv and ranks must be non-NULL");
  if (n_blocks < 1) return fail(MILO_ERR_INVALID_ARG, "n_blocks must be >= 1 (got %d)", n_blocks);
  if (ld < 1) return fail(MILO_ERR_INVALID_ARG, "ld must be >= 1");
  if (r_min < 0 || r_max < r_min)
    return fail(MILO_ERR_INVALID_ARG, "need 0 <= r_min <= r_max (got %d, %d)", r_min, r_max);
  std::vector<AllocBounds> bounds(n_blocks);
  int64_t floor_sum = 0, cand = 0;
  int32_t max_sv = 0;
  for (int b = 0; b < n_blocks; ++b) {
    if (n_sv[b] < 0 || n_sv[b] > ld)
      return fail(MILO_ERR_INVALID_ARG, "block %d: n_sv %d outside [0, ld=%lld]", b, n_sv[b], (long long)ld);
    AllocBounds& bd = bounds[b];
    bd.n_sv = n_sv[b];
    bd.lo = std::min(r_min, n_sv[b]);
    bd.hi = std::min(r_max, n_sv[b]);
    bd.pad = 0;
    floor_sum += bd.lo;
    cand += bd.hi - bd.lo;
    max_sv = std::max(max_sv, n_sv[b]);
  }
  if (r_total < floor_sum)
    return fail(MILO_ERR_INVALID_ARG, "budget %lld is below the sum of the floors %lld (no feasible allocation)",
                (long long)r_total, (long long)floor_sum);
  if (cand >= ((int64_t)1 << 31))
    return fail(MILO_ERR_UNSUPPORTED, "%lld candidate singular values exceed the supported 2^31", (long long)cand);
  const int32_t chunks = std::max(1, (max_sv + 255) / 256);
  if ((int64_t)n_blocks * chunks >= ((int64_t)1 << 31))
    return fail(MILO_ERR_UNSUPPORTED, "too many rows for one launch");
  // k units go to the largest candidates; none or all of them is the closed form
  // (floors or caps), but the values are still checked on the device
  const int64_t k = r_total - floor_sum;
  const bool select = k > 0 && k < cand;
  hipStream_t s = (hipStream_t)hip_stream;
  const size_t off_state = 0;  // workspace: state, bounds, counts, ranks
  const size_t st_bytes = (sizeof(AllocState) + 255) / 256 * 256;
  const size_t off_b = off_state + st_bytes;
  const size_t off_cnt = off_b + (size_t)n_blocks * sizeof(AllocBounds);
  const size_t off_rank = off_cnt + 2 * (size_t)n_blocks * sizeof(int32_t);
  const size_t total = off_rank + (size_t)n_blocks * sizeof(int32_t);
  char* ws = nullptr;
  MILO_HIP(hipMalloc((void**)&ws, total));
  hipEvent_t ev[10] = {};
  const bool timed = timing_enabled();
  bool queued = false;  // once work is queued, it must finish before the workspace is freed
  auto done = [&](int code) {
    if (queued) (void)hipStreamSynchronize(s);
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
    (void)hipFree(ws);
    return code;
  };
  hipError_t e;
  if (timed)
    for (hipEvent_t& x : ev)
      if ((e = hipEventCreate(&x)) != hipSuccess) return done(hip_fail(e, "hipEventCreate"));
  AllocArgs a{};
  a.sigma = sigma;
  a.ld = ld;
  a.n_blocks = n_blocks;
  a.chunks = chunks;
  a.bounds = (const AllocBounds*)(ws + off_b);
  a.st = (AllocState*)(ws + off_state);
  a.cnt = (int32_t*)(ws + off_cnt);
  a.ranks = (int32_t*)(ws + off_rank);
  queued = true;
  if ((e = hipMemcpyAsync(ws + off_b, bounds.data(), bounds.size() * sizeof(AllocBounds), hipMemcpyHostToDevice,
                          s)) != hipSuccess)
    return done(hip_fail(e, "hipMemcpyAsync(bounds)"));
  if ((e = launch_allocate(a, select ? (uint32_t)k : 0u, s, timed ? ev : nullptr)) != hipSuccess)
    return done(hip_fail(e, "allocation kernels"));
  int32_t bad = INT32_MAX;
  if ((e = hipMemcpyAsync(&bad, &a.st->bad_block, sizeof bad, hipMemcpyDeviceToHost, s)) != hipSuccess)
    return done(hip_fail(e, "hipMemcpyAsync(check)"));
  std::vector<int32_t> got(select ? n_blocks : 0);
  if (select && (e = hipMemcpyAsync(got.data(), a.ranks, got.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s)) !=
                    hipSuccess)
    return done(hip_fail(e, "hipMemcpyAsync(ranks)"));
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return done(hip_fail(e, "hipStreamSynchronize"));
  if (bad != INT32_MAX)
    return done(fail(MILO_ERR_INVALID_ARG,
                     "block %d: singular values must be finite, non-negative and non-increasing", bad));
  if (timed) {
    float chain = 0.f, hist = 0.f, t = 0.f;
    if ((e = hipEventElapsedTime(&chain, ev[0], ev[9])) != hipSuccess) return done(hip_fail(e, "hipEventElapsedTime"));
    for (int p = 0; p < (select ? 4 : 1); ++p) {
      if ((e = hipEventElapsedTime(&t, ev[1 + 2 * p], ev[2 + 2 * p])) != hipSuccess)
        return done(hip_fail(e, "hipEventElapsedTime"));
      hist += t;
    }
    std::lock_guard<std::mutex> lk(g_alloc_timing.mu);
    g_alloc_timing.chain_ms += chain;
    g_alloc_timing.hist_ms += hist;
    g_alloc_timing.calls += 1;
  }
  for (int b = 0; b < n_blocks; ++b) ranks[b] = select ? got[b] : (k == 0 ? bounds[b].lo : bounds[b].hi);
  return done(MILO_OK);
}

int milo_timing_read_alloc(double* chain_ms, double* hist_ms, int64_t* n_calls) {
  clear_error();
  std::lock_guard<std::mutex> lk(g_alloc_timing.mu);
  if (chain_ms) *chain_ms = g_alloc_timing.chain_ms;
  if (hist_ms) *hist_ms = g_alloc_timing.hist_ms;
  if (n_calls) *n_calls = g_alloc_timing.calls;
  g_alloc_timing.chain_ms = g_alloc_timing.hist_ms = 0.0;
  g_alloc_timing.calls = 0;
  return MILO_OK;
}

}  // extern "C"
