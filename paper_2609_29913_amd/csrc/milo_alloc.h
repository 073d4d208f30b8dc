// Internal interface of the entropy rank allocation (device side in
// milo_alloc.hip, host entry point milo_allocate_ranks there too).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace milo {

// Rank allocation (Sec. 4.3, Eqs. 5-7).  The greedy over marginal gains takes
// the k largest candidate singular values overall (each block's values are
// non-increasing and log(1 + x^2/eps^2) is increasing in x), equal values in
// block order; the device side finds the k-th largest value's bit pattern by a
// four-pass radix select (non-negative floats order like their bit patterns),
// then counts per block the candidates above it and hands the remaining units
// at that value out in block order.
constexpr int kHistCopies = 8;  // one histogram copy per XCD: workgroup b adds into copy b % 8

struct AllocState {
  uint32_t k;              // units to hand out beyond the floors
  int32_t bad_block;       // lowest block whose row breaks the precondition (INT32_MAX: none)
  uint32_t pad[62];
  uint32_t hist[4][kHistCopies][256];  // digit histogram of each radix pass (most significant first)
};

struct AllocBounds {
  int32_t n_sv;  // singular values in the row (all are checked)
  int32_t lo;    // the block's floor min(r_min, n_sv): candidates are columns lo .. hi-1
  int32_t hi;    // the block's cap min(r_max, n_sv)
  int32_t pad;
};

struct AllocArgs {
  const float* sigma;         // [n_blocks][ld] fp32, row b non-increasing in its first n_sv[b] columns
  int64_t ld;
  int32_t n_blocks;
  int32_t chunks;             // 256-column chunks per row (covers the longest row)
  const AllocBounds* bounds;  // [n_blocks]
  AllocState* st;
  int32_t* cnt;               // [2][n_blocks]: candidates above / equal to the selected key
  int32_t* ranks;             // [n_blocks]
};

// Queues the whole selection (k units over the candidates, 0 < k < candidates)
// or, with k == 0, only the state reset and the precondition check.  Each pass
// re-derives the digits picked so far from the earlier passes' histograms.  ev,
// when non-NULL, receives 10 events: chain start, (start, end) of each of the
// four histogram passes, chain end.
hipError_t launch_allocate(const AllocArgs& a, uint32_t k, hipStream_t s, hipEvent_t* ev);

}  // namespace milo
