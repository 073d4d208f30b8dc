// gfx950 (CDNA4) kernels for decode attention over a block-wise low-rank KV
// cache (MILO, Sec. 4.2 Eq. 3 factors; Sec. 4.4 Alg. 1 inference stage; the
// attention itself is Sec. 4.1 Eq. 1).
//
//  pack_kernel    repacks row-major bf16 factors into MFMA-fragment order.
//  attend_kernel  persistent: one workgroup (8 waves) per compute unit runs a
//                 host-built list of work items, its fragment streams flowing
//                 across items:
//     block item (block b, a tile of up to 64 head-major query columns of
//     one or more KV heads, a run of 256-token tiles):
//       projection  Qt = scale*log2(e) * R^K_b[:, g] q          (MFMA, into LDS;
//                   per KV head g of the tile)
//       scores      S  = P^K_b Qt, 32 tokens per wave and tile  (MFMA)
//       softmax     running max per column shared by the waves, W = 2^(S - m)
//       latent V    Ot = sum_t W_t P^V_b[t]                      (MFMA, waves split
//                   token segments x rank tiles)
//       up-project  o  = R^V_b[:, g]^T Ot                        (MFMA, 16-dim slice
//                   per wave; per KV head g of the tile)
//       -> folded into the workgroup's partial (m, l, o) per column for its
//          current column tile; written when the group ends
//     tail item (request i, KV head g, kTailChunk-token chunk of the request's
//     own KV): plain attention of the group's query heads over the chunk
//     (MFMA scores, VALU values) -> partial (m, l, o) per column
//  merge_kernel   log-sum-exp merge of every partial of a column into O (fp32).
//
// Scores are kept in log2 units (the scale folds log2(e)), so every exponential
// is one v_exp_f32.
#include <hip/hip_ext.h>

#include "milo_internal.h"

namespace milo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 ld_bf16x8(const void* p) { return *reinterpret_cast<const bf16x8*>(p); }

// eight int8 codes (little-endian in two dwords) as bf16, exactly
__device__ __forceinline__ bf16x8 i8_to_bf16x8(uint2 raw) {
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = (__bf16)(float)(int8_t)(raw.x >> (8 * e));
    v[4 + e] = (__bf16)(float)(int8_t)(raw.y >> (8 * e));
  }
  return v;
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// the same product on operands that hold fp16 bit patterns (rebuilt keys and
// the query of dense items)
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f32x16 mfma32_f16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// query row i * H_q + h of head-major column c = g * N_g + i * G + (h mod G)
__device__ __forceinline__ int64_t query_row(int c, int N_g, int G, int H_q) {
  const int g = c / N_g, rem = c - g * N_g, i = rem / G;
  return (int64_t)i * H_q + g * G + (rem - i * G);
}

// Direct global->LDS load of one fragment: lane l's 16 bytes from `src` land at
// LDS byte address lds_slot + 16 l.  Issued as inline assembly, so the compiler
// neither counts it nor orders other LDS accesses after it; every consumer
// waits for it explicitly (wait_vmcnt) before reading the slot.  M0 carries the
// slot address; no compiler-generated code in these kernels uses M0.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_slot) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_slot), "v"(src) : "memory");
}

// LDS reads of the workgroup's program (run lists, work items).  The compiler
// cannot tell these addresses from the slots that in-flight global->LDS loads
// write, so a plain LDS load here would make it wait for every outstanding
// fragment load; the program region is never a load target, so the reads are
// issued directly, waiting only for themselves.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>(p);  // offset within the LDS aperture
}
__device__ __forceinline__ int2 prog_read_b64(const void* p) {
  int2 v;
  asm volatile("ds_read_b64 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(lds_addr(p)));
  return v;
}
__device__ __forceinline__ int4 prog_read_b128(const void* p) {
  int4 v;
  asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(lds_addr(p)));
  return v;
}

// LDS stores the compiler would otherwise order after every in-flight
// global->LDS fragment load (it cannot prove they target other addresses).
__device__ __forceinline__ void lds_store_b128(void* p, float4 v) {
  const f32x4 x = {v.x, v.y, v.z, v.w};
  asm volatile("ds_write_b128 %0, %1" ::"v"(lds_addr(p)), "v"(x) : "memory");
}
__device__ __forceinline__ void lds_store_b64(void* p, int2 v) {
  asm volatile("ds_write_b64 %0, %1" ::"v"(lds_addr(p)), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_store_b32(void* p, float v) {
  asm volatile("ds_write_b32 %0, %1" ::"v"(lds_addr(p)), "v"(v) : "memory");
}

// Workgroup barrier for the attention kernel: every wave's LDS reads and
// writes issued before it are complete.  In-flight global->LDS fragment loads
// are deliberately not waited for (each targets its own wave's ring slots);
// __syncthreads() would make the compiler drain them (vmcnt(0)) at many
// barriers.  The "memory" clobber keeps the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (they complete in issue order).  The "memory" clobber keeps LDS reads of the
// slots it guards after it.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---------------------------------------------------------------------------
// Packing
// ---------------------------------------------------------------------------
// bf16 factor: the 8 elements of lane `lane` of fragment `frag`, one 16-byte store
__device__ __forceinline__ void pack_bf16_fragment(const PackArgs& a, int64_t frag, int lane) {
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    int row, col;
    frag_source(a.geom, frag, lane, e, &row, &col);
    v[e] = (row < a.geom.rows && col < a.geom.cols) ? a.src[(int64_t)row * a.geom.cols + col] : 0;
  }
  uint4 out;
  out.x = v[0] | ((uint32_t)v[1] << 16);
  out.y = v[2] | ((uint32_t)v[3] << 16);
  out.z = v[4] | ((uint32_t)v[5] << 16);
  out.w = v[6] | ((uint32_t)v[7] << 16);
  *reinterpret_cast<uint4*>(a.dst + frag * kFragElems + lane * 8) = out;
}

__global__ __launch_bounds__(256) void pack_kernel(PackArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t frag = gid >> 6;
  const int lane = (int)(gid & 63);
  if (frag >= a.n_frags) return;
  if (a.row_scale) {
    // INT8 P factor: code = round-to-nearest-even(P / s_row) in fp32 (correctly
    // rounded division), |code| <= 127; 8 codes per lane at byte 8 lane of the
    // fragment's 512 bytes
    uint32_t w[2] = {0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int row, col;
      frag_source(a.geom, frag, lane, e, &row, &col);
      int code = 0;
      if (row < a.geom.rows && col < a.geom.cols) {
        const float sc = a.row_scale[row];
        if (sc > 0.f) {
          const float x = bf16_to_f32(a.src[(int64_t)row * a.geom.cols + col]);
          code = (int)fminf(127.f, fmaxf(-127.f, rintf(__fdiv_rn(x, sc))));
        }
      }
      w[e >> 2] |= (uint32_t)(code & 0xff) << (8 * (e & 3));
    }
    *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(a.dst) + frag * kFragElems + lane * 8) =
        make_uint2(w[0], w[1]);
    return;
  }
  pack_bf16_fragment(a, frag, lane);
}

// Many bf16 factors in one launch: job j packs fragments
// starts[j] .. starts[j + 1] - 1 of a flat fragment range that begins at
// starts[0]; 4 fragments per workgroup, each lane finding its job by binary search.
__global__ __launch_bounds__(256) void pack_batch_kernel(const PackArgs* jobs, const int64_t* starts, int n_jobs) {
  const int64_t g = starts[0] + (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = (int)(threadIdx.x & 63);
  if (g >= starts[n_jobs]) return;
  int lo = 0, hi = n_jobs - 1;  // the last job whose start is <= g
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (starts[mid] <= g) lo = mid;
    else hi = mid - 1;
  }
  pack_bf16_fragment(jobs[lo], g - starts[lo], lane);
}

// INT8 P factors: per-row scale s = max |P[row][:]| / 127 (fp32, correctly
// rounded division); rows past `rows` up to rows_pad get 0; a non-finite row sets *bad.
__global__ __launch_bounds__(256) void row_scale_kernel(const uint16_t* src, int rows, int cols, int rows_pad,
                                                        float* scale, int* bad) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows_pad) return;
  float m = 0.f;
  if (r < rows) {
    for (int c = 0; c < cols; ++c) m = fmaxf(m, fabsf(bf16_to_f32(src[(int64_t)r * cols + c])));
    bool finite = true;
    for (int c = 0; c < cols; ++c) finite = finite && isfinite(bf16_to_f32(src[(int64_t)r * cols + c]));
    if (!finite) {
      atomicOr(bad, 1);
      m = 0.f;
    }
  }
  scale[r] = __fdiv_rn(m, 127.f);
}

// INT8 P factors: the 256-byte scale unit of (tile t, wave w) holds the K then
// the V scales of tokens 256 t + 32 w + m, m = 0..31
__global__ __launch_bounds__(256) void scale_units_kernel(const float* ks, const float* vs, int T_pad, float* dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;  // float index in the units
  if (i >= T_pad * 2) return;
  const int unit = i / 64, m = i % 64;                  // unit = t * kWaves + w
  const int tok = 32 * unit + (m & 31);
  dst[i] = m < 32 ? ks[tok] : vs[tok];
}

// ---------------------------------------------------------------------------
// Tail work item: attention of the G query heads of KV head g of request i over
// tokens [t0, t0 + nt) of that request's uncompressed KV (nt <= kTailChunk
// follows from the call's tail length; an item past the tail does nothing).  Wave w takes tokens t0 + 32w .. t0 + 32w + 31; every load of the
// item is issued up front (rows past the chunk's end re-read its last row and
// are masked), then:
//   scores  S = K q^T  (one 32x32x16 MFMA per 16 dims: 32 tokens x 32 head
//           columns, heads past G read the last head and are discarded)
//   softmax column max / sum over the 4 waves through LDS, W = 2^(S - m)
//   values  o[h] = sum_t W[t][h] V[t]  (VALU: lane owns D/64 dims, the weights
//           of a token are broadcast from LDS), summed over the waves in LDS.
// ---------------------------------------------------------------------------
// Value pass of a tail item for one wave: o[h][e] = sum over the wave's 32
// tokens of W[t][h] * V[t][e] for NH heads and this lane's D/64 dims, written
// to the wave's partial-output rows (row stride D).  Fully unrolled, so the
// per-token registers are addressed statically.
template <int D, int NH>
__device__ __forceinline__ void tail_values(const float* wt, const uint32_t (&vraw)[kTailChunk / kWaves],
                                            float* out) {
  constexpr int DL = D / 64;
  float acc[NH][DL];
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < DL; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int tt = 0; tt < kTailChunk / kWaves; ++tt) {
    float vf[DL];
    vf[0] = __uint_as_float(vraw[tt] << 16);
    if constexpr (DL == 2) vf[1] = __uint_as_float(vraw[tt] & 0xffff0000u);
    const float4* wr = reinterpret_cast<const float4*>(wt + tt * 32);
#pragma unroll
    for (int q4 = 0; q4 < NH / 4; ++q4) {
      const float4 w4 = wr[q4];
      const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < DL; ++e) acc[4 * q4 + u][e] += wv[u] * vf[e];
    }
  }
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < DL; ++e) out[h * D + e] = acc[h][e];
}

template <int D>
__device__ __forceinline__ void tail_item(const AttendArgs& a, const WorkItem& it, unsigned char* smem,
                                          const int tid) {
  constexpr int NK = D / 16;                // 16-dim steps of the score MFMA
  constexpr int DL = D / 64;                // dims per lane in the value pass
  constexpr int kTokW = kTailChunk / kWaves;  // tokens per wave (32)
  static_assert(kTokW == 32, "one 32-row MFMA tile of tokens per wave");
  const int i = it.req, slot = a.n_block_slots + it.slot, g = it.g, G = a.G;
  const int wave = tid >> 6, lane = tid & 63, lrow = lane & 31, lhi = lane >> 5;
  // the chunk's rows come from this call's tail length: the plan holds chunks
  // up to its planned capacity, and chunks past the request's tail are empty
  const int t0 = it.sub * kTailChunk;
  const int nt = min(kTailChunk, tail_len_of(a.tl, i) - t0);
  if (nt <= 0) return;
  float* red = reinterpret_cast<float*>(smem);   // [kWaves][32] column maxima
  float* lred = red + kWaves * 32;               // [kWaves][32] column sums
  float* wt = lred + kWaves * 32;                // [kTailChunk][32] weights, token-major
  float* op = wt + kTailChunk * 32;              // [kWaves][kMaxGroup][D] partial outputs

  const int64_t rs = (int64_t)a.H_kv * D;      // row stride of the tail K / V
  const int64_t row0 = (int64_t)i * a.tail_stride + t0;
  const int tk = min(kTokW * wave + lrow, nt - 1);   // this lane's token row (clamped)
  const int hh = min(lrow, G - 1);                    // this lane's head column (clamped)
  const uint16_t* krow = a.tail_k + (row0 + tk) * rs + (int64_t)g * D + 8 * lhi;
  const uint16_t* qrow = a.q + ((int64_t)i * a.H_q + g * G + hh) * D + 8 * lhi;
  const uint16_t* vcol = a.tail_v + row0 * rs + (int64_t)g * D + DL * lane;
  bf16x8 kf[NK], qf[NK];
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    kf[k] = ld_bf16x8(krow + 16 * k);
    qf[k] = ld_bf16x8(qrow + 16 * k);
  }
  uint32_t vraw[kTokW];  // V[token][DL*lane .. +DL-1] as bf16 bits
#pragma unroll
  for (int tt = 0; tt < kTokW; ++tt) {
    const int64_t r = min(kTokW * wave + tt, nt - 1);
    if constexpr (DL == 2) vraw[tt] = *reinterpret_cast<const uint32_t*>(vcol + r * rs);
    else vraw[tt] = vcol[r * rs];
  }
  // scores: lane holds head column lrow, token rows 8(v/4) + 4 lhi + v%4 of the wave's 32
  f32x16 sc = {};
#pragma unroll
  for (int k = 0; k < NK; ++k) sc = mfma32(kf[k], qf[k], sc);
  float mx = -INFINITY;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int tw = 8 * (v >> 2) + 4 * lhi + (v & 3);
    const float x = kTokW * wave + tw < nt ? sc[v] * a.qscale : -INFINITY;
    sc[v] = x;
    mx = fmaxf(mx, x);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  red[wave * 32 + lrow] = mx;  // both lane halves hold the same value
  lds_barrier();
  float m = red[lrow];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red[w * 32 + lrow]);
  float lsum = 0.f;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int tw = 8 * (v >> 2) + 4 * lhi + (v & 3);
    const float w = fast_exp2(sc[v] - m);  // masked tokens: 2^-inf = 0
    lsum += w;
    wt[(kTokW * wave + tw) * 32 + lrow] = w;
  }
  lsum += __shfl_xor(lsum, 32);
  lred[wave * 32 + lrow] = lsum;
  lds_barrier();
  // values over the wave's own tokens (heads rounded up to 8 or 16)
  if (G <= 8) tail_values<D, 8>(wt + kTokW * wave * 32, vraw, op + wave * kMaxGroup * D + DL * lane);
  else tail_values<D, kMaxGroup>(wt + kTokW * wave * 32, vraw, op + wave * kMaxGroup * D + DL * lane);
  lds_barrier();
  for (int x = tid; x < G * D; x += kThreads) {
    const int h = x / D, dd = x % D;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) o += op[(w * kMaxGroup + h) * D + dd];
    const int64_t col = (int64_t)i * a.H_q + g * G + h;
    a.part_o[(col * a.n_slots + slot) * D + dd] = o;
    if (dd == 0) {
      float mm = red[h], ll = 0.f;
#pragma unroll
      for (int w = 1; w < kWaves; ++w) mm = fmaxf(mm, red[w * 32 + h]);
#pragma unroll
      for (int w = 0; w < kWaves; ++w) ll += lred[w * 32 + h];
      a.part_ml[col * a.n_slots + slot] = make_float2(mm, ll);
    }
  }
}

// a work item read from LDS into wave-uniform registers
__device__ __forceinline__ WorkItem lds_item(const unsigned char* p) {
  static_assert(sizeof(WorkItem) == 80, "a work item is five 16-byte chunks");
  int4 v0, v1, v2, v3, v4;
  const uint32_t a = lds_addr(p);
  asm volatile(
      "ds_read_b128 %0, %5\n\tds_read_b128 %1, %5 offset:16\n\tds_read_b128 %2, %5 offset:32\n\t"
      "ds_read_b128 %3, %5 offset:48\n\tds_read_b128 %4, %5 offset:64\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(v0), "=&v"(v1), "=&v"(v2), "=&v"(v3), "=&v"(v4)  // early clobber: the address
      : "v"(a));                                                // must survive the first reads
  const int4 vv[5] = {v0, v1, v2, v3, v4};
  int32_t w[20];
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    w[4 * i + 0] = __builtin_amdgcn_readfirstlane(vv[i].x);
    w[4 * i + 1] = __builtin_amdgcn_readfirstlane(vv[i].y);
    w[4 * i + 2] = __builtin_amdgcn_readfirstlane(vv[i].z);
    w[4 * i + 3] = __builtin_amdgcn_readfirstlane(vv[i].w);
  }
  WorkItem it;
  __builtin_memcpy(&it, w, sizeof(WorkItem));
  return it;
}

// A wave's fragment stream over all block items of its workgroup: the runs of
// consecutive packed fragments in the order the wave consumes them (per block
// item: its R^K run for the projection, then for every 256-token tile its P^K
// run and its P^V run, then its R^V run for the up-projection; block_runs).
// Wave 0 derives them item by item for all waves (RunDeriver below) into four
// LDS run buffers per wave used in turn (entry (x, n): n consecutive fragments
// from fragment x; (x, 0) ends a buffer), staying two block items ahead of the
// item being computed: every item gives every wave at least three fragments
// and the look-ahead loads run at most kDepth <= 6 fragments ahead, so they
// never reach a buffer that is not ready, and the buffer being refilled is two
// items behind.  Runs are read when their first fragment is issued.  After the
// last block item a long sentinel run follows.  With NSLOT > 0 fragments reach the wave through a private ring of NSLOT LDS
// slots, filled by direct global->LDS loads issued kDepth fragments ahead of
// use, so every wait is a constant vmcnt; the look-ahead crosses item
// boundaries, so the next item's first fragments load while the current one
// finishes.  With NSLOT == 0 fragments are loaded straight into registers.
template <int D, int NSLOT, bool I8>
struct FragRing {
  static constexpr int kDepth = NSLOT > 2 ? NSLOT - 2 : 1;  // units in flight
  static_assert(kDepth <= 6, "run buffers are derived two block items (>= 6 units) ahead");
  const unsigned char* data;  // packed factor buffer
  int lane;                   // this lane
  __bf16* ring;               // this wave's NSLOT slots
  uint32_t ring_lds;          // LDS byte address of slot 0 (wave-uniform)
  const int2* run;            // current entry of the run buffers (LDS)
  int2* rbuf;                 // this wave's kRunBufs run buffers of run_cap entries
  int run_cap;
  int rb;                     // buffer the stream reads
  int64_t off;                // byte offset of the next unit
  int left;                   // units left in the current run
  int step;                   // bytes per unit of the current run (1 KiB, or 256 for scale units)
  int lane_off;               // this lane's byte offset in a unit of the current run
  int rs, ws;                 // ring slots: next to read, next to fill
  bf16x8 held;                // the second fragment of the last int8 unit taken
  bool have_held;

  __device__ __forceinline__ void load_run() {
    int2 v = prog_read_b64(run);
    if (__builtin_amdgcn_readfirstlane(v.y) == 0) {  // end of a buffer: the next one
      rb = (rb + 1) % kRunBufs;
      run = rbuf + rb * run_cap;
      v = prog_read_b64(run);
    }
    const int x = __builtin_amdgcn_readfirstlane(v.x), n = __builtin_amdgcn_readfirstlane(v.y);
    if constexpr (!I8) {  // every run holds bf16 fragments
      off = (int64_t)x * (kFragElems * 2);
      left = n;
      return;
    }
    const int kind = (n >> kRunKindShift) & 3, count = n & kRunCountMask;
    if (kind == kRunBf16) {
      off = (int64_t)x * (kFragElems * 2);
      left = count;
      step = kFragElems * 2;
      lane_off = 16 * lane;
    } else if (kind == kRunI8) {  // two 512-byte fragments per unit
      off = (int64_t)x * (kFragElems);
      left = count >> 1;
      step = kFragElems * 2;
      lane_off = 16 * lane;
    } else {  // scale unit: 256 bytes, every group of 16 lanes loads all of it
      off = (int64_t)x * kScaleUnitBytes;
      left = count;
      step = kScaleUnitBytes;
      lane_off = 16 * (lane & 15);
    }
  }
  // the unit's start, and this lane's address in the next unit; advances the stream
  __device__ __forceinline__ const unsigned char* next(const unsigned char** unit = nullptr) {
    if (left == 0) {
      ++run;
      load_run();
    }
    const unsigned char* u = data + off;
    if (unit) *unit = u;
    --left;
    if constexpr (!I8) {
      off += kFragElems * 2;
      return u + 16 * lane;
    } else {
      off += step;
      return u + lane_off;
    }
  }
  __device__ __forceinline__ void start() {
    rb = 0;
    run = rbuf;
    load_run();
    rs = 0;
    ws = 0;
    have_held = false;
    if constexpr (NSLOT > 0) {
#pragma unroll
      for (int k = 0; k < kDepth; ++k) lds_dma16(next(), ring_lds + k * kFragElems * 2);
      ws = kDepth;
    }
  }
  // the slot (LDS) or unit (global memory) of the next unit, and advance
  __device__ __forceinline__ const unsigned char* next_unit() {
    if constexpr (NSLOT > 0) {
      wait_vmcnt<kDepth - 1>();
      const unsigned char* slot = reinterpret_cast<const unsigned char*>(ring + rs * kFragElems);
      lds_dma16(next(), ring_lds + ws * kFragElems * 2);
      rs = rs + 1 == NSLOT ? 0 : rs + 1;
      ws = ws + 1 == NSLOT ? 0 : ws + 1;
      return slot;
    } else {
      const unsigned char* u;
      next(&u);
      return u;
    }
  }
  // the next bf16 fragment, in this lane's operand layout
  __device__ __forceinline__ bf16x8 take() {
    return ld_bf16x8(next_unit() + 16 * lane);
  }
  // the next fragment of an int8 run, converted to bf16 (exact: |code| <= 127);
  // a unit holds two fragments, the second is kept for the following call
  __device__ __forceinline__ bf16x8 take_i8() {
    static_assert(I8, "int8 fragments only in the INT8 instantiation");
    if (have_held) {
      have_held = false;
      return held;
    }
    const unsigned char* u = next_unit();
    const uint2 lo = *reinterpret_cast<const uint2*>(u + 8 * lane);
    const uint2 hi = *reinterpret_cast<const uint2*>(u + kFragElems + 8 * lane);
    held = i8_to_bf16x8(hi);
    have_held = true;
    return i8_to_bf16x8(lo);
  }
  // the next scale unit: 32 K then 32 V scales (fp32); the pointer stays valid
  // until the next take
  __device__ __forceinline__ const float* take_scales() {
    return reinterpret_cast<const float*>(next_unit());
  }
};

// Derivation of the fragment runs, done by wave 0 for all eight waves (lane w
// derives wave w's runs, in vector registers): the runs of the workgroup's
// next block item, or the sentinel run after the last one, into every wave's
// buffer gb.  Runs are read by their wave only after a later workgroup
// barrier.
template <int D>
struct RunDeriver {
  const unsigned char* items;  // the workgroup's work items (LDS)
  int n_items;
  int gk;                      // next item to look at
  int gb;                      // buffer the next derivation fills
  int2* rbuf;                  // all waves' run buffers: [wave][kRunBufs][run_cap]
  int run_cap;
  int recon_delta;             // fragments from the factor buffer to the reconstruction buffer

  __device__ void derive(int lane) {
    WorkItem it{};
    bool found = false;
    while (gk < n_items) {
      it = lds_item(items + (size_t)gk * sizeof(WorkItem));
      ++gk;
      if (it.kind == kItemBlock) {
        found = true;
        break;
      }
    }
    if (lane < kWaves) {
      int2* out = rbuf + ((size_t)lane * kRunBufs + gb) * run_cap;
      int n = 0;
      auto put = [&](int x, int cnt) {
        lds_store_b64(out + n, make_int2(x, cnt));
        ++n;
      };
      if (found)
        block_runs(it.blk, it.g, ((it.flags >> kItemHeadsShift) & 7) + 1, it.tile0, it.ntile, lane, D,
                   (it.flags >> kItemLgNgShift) & 3, (it.flags & kItemInt8) != 0, put, (it.flags & kItemDense) != 0,
                   recon_delta);
      else put(0, kSentinelRun);
      put(0, 0);
    }
    gb = (gb + 1) % kRunBufs;
  }
};

// A workgroup's running partial for its current group of block items (one KV
// head and column tile): the output in the up-projection's lane layout (NCB
// 16-column blocks of the wave's 16-dim slice), the per-column maximum in the
// score layout (32 ch + lane % 32; every wave holds it), the per-column sum
// in wave 0 (thread t: column t).
template <int NCB>
struct GroupAcc {
  f32x4 o[NCB];
  float m[2];
  float l;
};
template <int D>
constexpr int up_col_blocks() {
  return 4 * (D / 16) / kWaves;  // 16-column blocks per wave in the up-projection
}

// ---------------------------------------------------------------------------
// Block work item: latent-space attention of one column tile (at most 64
// consecutive head-major query columns, of up to kMaxTileHeads KV heads) over
// the tiles [tile0, tile0 + ntile) of block b.  The scores and the latent
// value pass do not depend on the head (P^K and P^V are shared by all KV
// heads); the projection and the up-projection run once per KV head of the
// tile, each column keeping the result of its own head.
//
// Eight waves (two per SIMD).  Scores: wave w takes the 32 tokens 32w..32w+31
// of every 256-token tile against all 64 columns.  Latent V: the waves form
// nseg token segments x ng rank groups (see the packed layout), so each wave
// accumulates its own rank tiles over its own tokens; the segments' partial
// sums are then combined in LDS and the latent result goes to LDS as bf16.
// Up-projection: each wave computes a 16-dim slice of the output for all 64
// columns over all ranks.  Every factor fragment a wave consumes (R^K for the
// projection, P^K and P^V per tile, R^V for the up-projection) comes from the
// wave's fragment stream (FragRing above); the item's queries are loaded into
// LDS at its start.  Every loop is software-pipelined: the operands of step
// k+1 are read while the MFMAs of step k run.
// ---------------------------------------------------------------------------
// MODE: 0 bf16 P factors, 1 INT8 P factors, 2 bf16 P factors with the
// projection as a wavefront GEMV (kernel variants, so no branch of one costs
// the others registers)
template <int D, int MAX_RT, int NSLOT, bool WH, int MODE>
__device__ __forceinline__ void block_item(const AttendArgs& a, const WorkItem& it, unsigned char* smem,
                                           FragRing<D, NSLOT, MODE == 1>& fr, RunDeriver<D>& rd,
                                           GroupAcc<up_col_blocks<D>()>& acc, const int tid) {
  constexpr bool I8 = MODE == 1, GV = MODE == 2;
  constexpr int NK = D / 16;
  constexpr int kORed = 4;  // partial-output slots of the up-projection reduction
  const BlockMeta& bm = it.blk;
  const int slot = it.slot, g0 = it.g, c0 = it.req;
  const int cn = ((it.flags >> kItemColsShift) & 63) + 1;  // columns of the tile
  const int nh = ((it.flags >> kItemHeadsShift) & 7) + 1;  // KV heads of the tile
  // a reconstructed block: bm names K_{b,g} / V_{b,g} of the tile's one KV head
  // (rank d); the query takes the projection's place and the value pass gives
  // the output
  const bool dense = (it.flags & kItemDense) != 0;
  const bool causal = (it.flags & kItemCausal) != 0;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 31, lhi = lane >> 5;
  const int G = a.G, N_g = a.N_g;
  const int qsd = a.qt_stride;
  const int nrt_k = bm.rk_pad >> 5, nks = bm.rk_pad >> 4;
  const int nrt_v = bm.rv_pad >> 5;
  const int own_k = owned_tiles(nrt_k, wave, kWaves);
  const int nseg = v_segments(nrt_v), ng = kWaves / nseg;
  const int rg = wave % ng, sg = wave / ng;
  const int own_v = owned_tiles(nrt_v, rg, ng);
  const int nst = 16 / nseg;                // 16-token steps of the wave's segment per tile
  const int T = bm.T;
  const int ntiles = it.ntile, tile0 = it.tile0;  // tiles this item covers
  // causal limits of this lane's two columns (32 ch + lane % 32; request (c mod N_g) / G)
  // and the smallest over the tile (wave-uniform), past which tokens need masking
  int lim[2] = {T, T}, lim_min = T;
  if (causal) {
#pragma unroll
    for (int ch = 0; ch < 2; ++ch)
      lim[ch] = tail_len_of(a.tl, ((c0 + min(32 * ch + (lane & 31), cn - 1)) % N_g) / G);
    lim_min = min(lim[0], lim[1]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) lim_min = min(lim_min, __shfl_xor(lim_min, off));
  }
  __bf16* qt = reinterpret_cast<__bf16*>(smem);              // [kCols][qsd]
  // the weight tile: [kCols][kWS] bf16, all 256 tokens of a tile, or (WH) one
  // 128-token half at a time when LDS is short (ranks above 512)
  constexpr int kWS = WH ? kTile / 2 + 8 : kWStride;
  __bf16* wl = qt + kCols * qsd;                          // [kCols][kWS]
  float* red = reinterpret_cast<float*>(wl + kCols * kWS);  // [kWaves][kCols]
  // the wave's next fragment; the order of take() calls below is the order of
  // the wave's runs: R^K (waves that own projection rank tiles), then per tile
  // P^K and P^V, then R^V
  auto take = [&]() -> bf16x8 { return fr.take(); };
  // P^K / P^V fragments: bf16, or int8 codes converted exactly (INT8 P factors)
  auto take_p = [&]() -> bf16x8 {
    if constexpr (I8) return fr.take_i8();
    else return fr.take();
  };

  // ---- the item's 64 query rows -> LDS (in the weight tile's area, idle until
  // the first tile).  Row-major [column][D]; the 16-byte chunk j of column c is
  // stored at chunk position j ^ (c % kRowChunks), so the projection's operand
  // reads (same chunk, 32 columns) hit distinct banks.  Columns past the tile's
  // last one re-read the last column's query and count as its head (their
  // results are never stored).
  constexpr int kRowChunks = D / 8;              // 16-byte chunks per query row
  constexpr int kRowsPerLoad = 64 / kRowChunks;  // rows per 1 KiB load
  const __bf16* qimg = wl;
  {
    const uint32_t qimg_lds = __builtin_amdgcn_readfirstlane(lds_addr(qimg));
    const int cl_lane = lane / kRowChunks, pos = lane % kRowChunks;
    for (int f = wave; f < kCols / kRowsPerLoad; f += kWaves) {
      const int cl = kRowsPerLoad * f + cl_lane;
      const uint16_t* src = a.q + query_row(c0 + min(cl, cn - 1), N_g, G, a.H_q) * D + 8 * (pos ^ (cl % kRowChunks));
      lds_dma16(src, qimg_lds + f * 1024);
    }
    if (wave == 0) rd.derive(lane);  // the runs of the block item two ahead, while the rows load
    wait_vmcnt<0>();
    lds_barrier();
  }

  // ---- projection: Qt[rank][col] (stored [col][rank]), once per KV head of
  // the tile; each column stores its own head's result.  Dense items: Qt is
  // the query itself times the sign of the scale, as fp16 (exact for the
  // bf16 query in fp16's normal range; saturated at +-65504) to meet the
  // rebuilt keys, which are fp16 too, in the fp16 score MFMA; the scale's
  // magnitude goes onto the fp32 scores (sscale below).  A scaled query
  // rounded to 16 bits would put a relative rounding error on every score,
  // which a peaked softmax magnifies ----
  if (dense) {
    const float sgn = a.qscale > 0.f ? 1.f : a.qscale < 0.f ? -1.f : 0.f;
    for (int x = tid; x < kCols * kRowChunks; x += kThreads) {
      const int cl = x / kRowChunks, j = x % kRowChunks;
      const bf16x8 v = ld_bf16x8(qimg + cl * D + 8 * (j ^ (cl % kRowChunks)));
      f16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (_Float16)fminf(fmaxf((float)v[e] * sgn, -65504.f), 65504.f);
      *reinterpret_cast<f16x8*>(qt + cl * qsd + 8 * j) = o;
    }
  } else if (GV && own_k > 0) {
    // small batches (a tile of at most kGemvCols columns): the projection as a
    // wavefront GEMV.  Lane (c, m) of an R^K fragment holds rank 32 rt + m, dims
    // 16 k + 8 c .. +7; it dots them with the same dims of every column of the
    // current head (the query row chunk is one LDS broadcast), the two lane
    // halves are summed, and lanes m < 32 store their rank of the head's columns.
    // Columns past the tile's last one get zeros.
    for (int x = 0; x < nh * own_k; ++x) {
      const int hh = x / own_k, rt = wave + kWaves * (x - hh * own_k);
      // the head's columns are the consecutive range [lo, hi) of the tile
      const int lo = max(0, (g0 + hh) * N_g - c0), hi = min(cn, (g0 + hh + 1) * N_g - c0);
      float acc[kGemvCols];
#pragma unroll
      for (int cl = 0; cl < kGemvCols; ++cl) acc[cl] = 0.f;
      for (int k = 0; k < NK; ++k) {
        const bf16x8 af = take();
        float rf[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) rf[e] = (float)af[e];
        // every one of the kGemvCols query rows (rows past the tile's columns
        // hold a copy of its last one); only the head's columns are stored
#pragma unroll
        for (int cl = 0; cl < kGemvCols; ++cl) {
          const bf16x8 qv = ld_bf16x8(qimg + cl * D + 8 * ((2 * k + lhi) ^ (cl % kRowChunks)));
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[cl] = fmaf(rf[e], (float)qv[e], acc[cl]);
        }
      }
#pragma unroll
      for (int cl = 0; cl < kGemvCols; ++cl) {
        acc[cl] += __shfl_xor(acc[cl], 32);
        if (lhi == 0 && cl >= lo && cl < hi) qt[cl * qsd + 32 * rt + lrow] = (__bf16)(acc[cl] * a.qscale);
      }
      if (hh == 0)
        for (int cl = cn + lhi; cl < kCols; cl += 2) qt[cl * qsd + 32 * rt + lrow] = (__bf16)0.f;
    }
  } else if (own_k > 0) {
    bf16x8 qf[NK][2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch)
#pragma unroll
      for (int k = 0; k < NK; ++k)
        qf[k][ch] = ld_bf16x8(qimg + (32 * ch + lrow) * D + 8 * ((2 * k + lhi) ^ (lrow % kRowChunks)));
    // KV head (relative to g0) of this lane's two columns 32 ch + lrow
    const int hq0 = (c0 + min(lrow, cn - 1)) / N_g - g0;
    const int hq1 = (c0 + min(32 + lrow, cn - 1)) / N_g - g0;
    for (int x = 0; x < nh * own_k; ++x) {
      const int hh = x / own_k, rt = wave + kWaves * (x - hh * own_k);
      f32x16 acc0 = {}, acc1 = {};
      bf16x8 af = take();
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        bf16x8 an = af;
        if (k + 1 < NK) an = take();
        acc0 = mfma32(af, qf[k][0], acc0);
        acc1 = mfma32(af, qf[k][1], acc1);
        af = an;
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        bf16x4 v0, v1;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          v0[u] = (__bf16)(acc0[4 * jj + u] * a.qscale);
          v1[u] = (__bf16)(acc1[4 * jj + u] * a.qscale);
        }
        const int r = 32 * rt + 8 * jj + 4 * lhi;
        if (hq0 == hh) *reinterpret_cast<bf16x4*>(qt + lrow * qsd + r) = v0;
        if (hq1 == hh) *reinterpret_cast<bf16x4*>(qt + (32 + lrow) * qsd + r) = v1;
      }
    }
  }
  lds_barrier();

  // ---- scores, online softmax, latent V ----
  f32x16 oacc[MAX_RT][2];
#pragma unroll
  for (int r = 0; r < MAX_RT; ++r) oacc[r][0] = oacc[r][1] = f32x16{};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};
  // factor (> 0) from the MFMA's raw scores to scores in log2 units: the
  // magnitude of the scale for dense items, 1 otherwise (the projection
  // carries it); applied in the column maximum and the weights' exponent
  const float sscale = dense && a.qscale != 0.f ? fabsf(a.qscale) : 1.f;
  const __bf16* qr0 = qt + lrow * qsd + 8 * lhi;
  const __bf16* qr1 = qt + (32 + lrow) * qsd + 8 * lhi;
  // weight operand rows of the wave's segment (relative step st at 16 st)
  const __bf16* wr0 = wl + lrow * kWS + 8 * lhi + 16 * nst * sg;
  const __bf16* wr1 = wl + (32 + lrow) * kWS + 8 * lhi + 16 * nst * sg;

  for (int tt = 0; tt < ntiles; ++tt) {
    const int tw = (tile0 + tt) * kTile + wave * kTokWave;
    f32x16 s0 = {}, s1 = {};
    // operands of rank step k: ak (P^K sub-tile, or rebuilt keys), b0/b1 (Qt
    // column tiles); nks is even (ranks are padded to 32), so the loop runs over
    // step pairs; dense items multiply fp16 operands
    auto scores = [&](auto mma) {
      bf16x8 ak = take_p();
      bf16x8 b0 = ld_bf16x8(qr0), b1 = ld_bf16x8(qr1);
      for (int k = 0; k < nks; k += 2) {
        const bf16x8 ck = take_p();
        const bf16x8 d0 = ld_bf16x8(qr0 + 16 * (k + 1));
        const bf16x8 d1 = ld_bf16x8(qr1 + 16 * (k + 1));
        s0 = mma(ak, b0, s0);
        s1 = mma(ak, b1, s1);
        if (k + 2 < nks) {
          ak = take_p();
          b0 = ld_bf16x8(qr0 + 16 * (k + 2));
          b1 = ld_bf16x8(qr1 + 16 * (k + 2));
        }
        s0 = mma(ck, d0, s0);
        s1 = mma(ck, d1, s1);
      }
    };
    if constexpr (I8) {
      scores(mfma32);
    } else {
      if (dense) scores(mfma32_f16);
      else scores(mfma32);
    }
    f32x16 sc[2] = {s0, s1};
    // INT8 P factors: the scores of int8 codes times each token's K scale; the
    // V scales fold into the weights below (lane: tokens 8 j + 4 lhi + u of the
    // wave's 32, j, u = 0..3)
    float vsc[16];
    if constexpr (I8) {
      const float* su = fr.take_scales();
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 k4 = *reinterpret_cast<const float4*>(su + 8 * j + 4 * lhi);
        const float4 v4 = *reinterpret_cast<const float4*>(su + 32 + 8 * j + 4 * lhi);
        const float kk[4] = {k4.x, k4.y, k4.z, k4.w}, vv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          sc[0][4 * j + u] *= kk[u];
          sc[1][4 * j + u] *= kk[u];
          vsc[4 * j + u] = vv[u];
        }
      }
    }
    // mask tokens past the end of the block (only the block's last tile can
    // hold any; the test is wave-uniform), and for a prefill chunk's shared
    // tail the tokens past each column's causal limit; wave-local column max
    float mx[2] = {-INFINITY, -INFINITY};
    if (tw + kTokWave > T || (causal && tw + kTokWave > lim_min)) {
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int tok = tw + 8 * (v >> 2) + 4 * lhi + (v & 3);
          if (tok >= T || tok >= lim[ch]) sc[ch][v] = -INFINITY;
        }
    }
#pragma unroll
    for (int ch = 0; ch < 2; ++ch)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx[ch] = fmaxf(mx[ch], sc[ch][v]);
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      mx[ch] = fmaxf(mx[ch], __shfl_xor(mx[ch], 32)) * sscale;
      red[wave * kCols + 32 * ch + lrow] = mx[ch];  // both lane halves hold the same value
    }
    lds_barrier();
    float alpha[2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      float tm = red[32 * ch + lrow];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) tm = fmaxf(tm, red[w * kCols + 32 * ch + lrow]);
      const float mn = fmaxf(m_run[ch], tm);
      // a column with no key so far (a causal column before its first token)
      // keeps m = -inf and zero weights
      alpha[ch] = mn == -INFINITY ? 1.f : fast_exp2(m_run[ch] - mn);
      m_run[ch] = mn;
    }
    // weights W = 2^(s - m) (bf16) in registers, then to LDS as [col][token]
    bf16x4 wv[2][4];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      float lsum = 0.f;
      const float mref = m_run[ch] == -INFINITY ? 0.f : m_run[ch];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float w = fast_exp2(fmaf(sc[ch][4 * j + u], sscale, -mref));
          lsum += w;
          if constexpr (I8) wv[ch][j][u] = (__bf16)(w * vsc[4 * j + u]);
          else wv[ch][j][u] = (__bf16)w;
        }
      l_run[ch] = l_run[ch] * alpha[ch] + lsum;
    }
    auto write_w = [&]() {
      const int tcol = (WH ? (wave & 3) : wave) * kTokWave;  // the wave's tokens in the (half) tile
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<bf16x4*>(wl + (32 * ch + lrow) * kWS + tcol + 8 * j + 4 * lhi) = wv[ch][j];
    };
    // latent V over the wave's relative steps [lo, hi) (even bounds), weights
    // of relative step st at w0p / w1p + 16 st
    auto vpass = [&](int lo, int hi, const __bf16* w0p, const __bf16* w1p) {
      if (own_v <= 0 || lo >= hi) return;
      // operands of 16-token step st: w0/w1 (weight column tiles), pa[r] (P^V rank
      // tiles); the loop runs over step pairs
      bf16x8 pa[MAX_RT], pc[MAX_RT];
      bf16x8 w0 = ld_bf16x8(w0p + 16 * lo), w1 = ld_bf16x8(w1p + 16 * lo);
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r)
        if (r < own_v) pa[r] = take_p();
      for (int st = lo; st < hi; st += 2) {
        const bf16x8 x0 = ld_bf16x8(w0p + 16 * (st + 1));
        const bf16x8 x1 = ld_bf16x8(w1p + 16 * (st + 1));
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v) pc[r] = take_p();
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v) {
            oacc[r][0] = mfma32(pa[r], w0, oacc[r][0]);
            oacc[r][1] = mfma32(pa[r], w1, oacc[r][1]);
          }
        if (st + 2 < hi) {
          w0 = ld_bf16x8(w0p + 16 * (st + 2));
          w1 = ld_bf16x8(w1p + 16 * (st + 2));
#pragma unroll
          for (int r = 0; r < MAX_RT; ++r)
            if (r < own_v) pa[r] = take_p();
        }
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v) {
            oacc[r][0] = mfma32(pc[r], x0, oacc[r][0]);
            oacc[r][1] = mfma32(pc[r], x1, oacc[r][1]);
          }
      }
    };
    auto rescale = [&]() {
      // rescale the latent accumulators to the new running maximum; skipped on
      // the first tile (they are zero) and when no column's maximum moved
      if (tt > 0 && own_v > 0 && __any(alpha[0] != 1.f || alpha[1] != 1.f)) {
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v) {
            oacc[r][0] *= alpha[0];
            oacc[r][1] *= alpha[1];
          }
      }
    };
    if constexpr (!WH) {
      write_w();
      lds_barrier();
      rescale();
      vpass(0, nst, wr0, wr1);
    } else {
      // half h holds the tokens of waves 4h .. 4h+3, i.e. tile steps [8h, 8h + 8);
      // the wave's segment covers tile steps [nst sg, nst sg + nst)
      if (wave < 4) write_w();
      lds_barrier();
      rescale();
      vpass(0, min(nst, 8 - nst * sg), wr0, wr1);
      lds_barrier();  // every wave is done with the first half's weights
      if (wave >= 4) write_w();
      lds_barrier();
      vpass(max(0, 8 - nst * sg), nst, wr0 - 16 * 8, wr1 - 16 * 8);
    }
  }

  // ---- up-projection through R^V and the partial (m, l, o) ----
#pragma unroll
  for (int ch = 0; ch < 2; ++ch) l_run[ch] += __shfl_xor(l_run[ch], 32);
  lds_barrier();  // every wave is done with qt / wl
  float* lred = reinterpret_cast<float*>(smem + a.ring_offset) - kWaves * kCols;  // [kWaves][kCols]
  lred[wave * kCols + lrow] = l_run[0];  // both lane halves hold the sums
  lred[wave * kCols + 32 + lrow] = l_run[1];
  // combine the token segments' latent partials (pairwise rounds through LDS,
  // fp32): the waves of segments [h, 2h) hand theirs to segments [0, h)
  if (nseg > 1) {
    float* segbuf = reinterpret_cast<float*>(smem);  // [slot][owned tile][ch][16][64 lanes]
    const int own_max = (nrt_v + ng - 1) / ng;        // slot size: the largest rank group's tiles
    for (int h = nseg / 2; h >= 1; h /= 2) {
      if (sg >= h && sg < 2 * h) {
        float* dst = segbuf + (int64_t)((sg - h) * ng + rg) * own_max * 2 * 16 * 64 + lane;
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v)
#pragma unroll
            for (int ch = 0; ch < 2; ++ch)
#pragma unroll
              for (int v = 0; v < 16; ++v) dst[((r * 2 + ch) * 16 + v) * 64] = oacc[r][ch][v];
      }
      lds_barrier();
      if (sg < h) {
        const float* src = segbuf + (int64_t)(sg * ng + rg) * own_max * 2 * 16 * 64 + lane;
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < own_v)
#pragma unroll
            for (int ch = 0; ch < 2; ++ch)
#pragma unroll
              for (int v = 0; v < 16; ++v) oacc[r][ch][v] += src[((r * 2 + ch) * 16 + v) * 64];
      }
      lds_barrier();
    }
  }
  constexpr int NDS = D / 16;              // 16-dim slices
  constexpr int NCB = up_col_blocks<D>();  // 16-column blocks per wave
  const int ds = wave % NDS, cb0 = (wave / NDS) * NCB;
  f32x4 uacc[NCB];
  if (dense) {
    // the value pass already produced the output: its accumulators (fp32,
    // [col][dim]) through LDS into the up-projection's lane layout
    float* of = reinterpret_cast<float*>(smem);
    constexpr int ofs = D + 4;
    if (sg == 0) {
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r)
        if (r < own_v) {
          const int rt = rg + ng * r;
#pragma unroll
          for (int ch = 0; ch < 2; ++ch)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
              *reinterpret_cast<float4*>(of + (32 * ch + lrow) * ofs + 32 * rt + 8 * jj + 4 * lhi) =
                  make_float4(oacc[r][ch][4 * jj], oacc[r][ch][4 * jj + 1], oacc[r][ch][4 * jj + 2],
                              oacc[r][ch][4 * jj + 3]);
        }
    }
    lds_barrier();
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const float4 v = *reinterpret_cast<const float4*>(of + (16 * (cb0 + cb) + (lane & 15)) * ofs + 16 * ds +
                                                        4 * (lane >> 4));
      uacc[cb] = f32x4{v.x, v.y, v.z, v.w};
    }
  } else {
    // the latent accumulator of every rank tile -> LDS as bf16 [col][rank]
    __bf16* olat = reinterpret_cast<__bf16*>(smem);
    const int ols = bm.rv_pad + 8;
    if (sg == 0) {
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r)
        if (r < own_v) {
          const int rt = rg + ng * r;
#pragma unroll
          for (int ch = 0; ch < 2; ++ch)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              bf16x4 v;
#pragma unroll
              for (int u = 0; u < 4; ++u) v[u] = (__bf16)oacc[r][ch][4 * jj + u];
              *reinterpret_cast<bf16x4*>(olat + (32 * ch + lrow) * ols + 32 * rt + 8 * jj + 4 * lhi) = v;
            }
        }
    }
    lds_barrier();
    // every wave: output dims [16 ds, 16 ds + 16) of its 16-column blocks, over
    // all ranks (16x16x32 MFMAs: R^V fragment x latent columns from LDS)
    {
      // KV head (relative to g0) of this lane's output columns
      int hu[NCB];
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) hu[cb] = (c0 + min(16 * (cb0 + cb) + (lane & 15), cn - 1)) / N_g - g0;
      const int nk = bm.rv_pad >> 5;
      const __bf16* ob = olat + (16 * cb0 + (lane & 15)) * ols + 8 * (lane >> 4);
      for (int hh = 0; hh < nh; ++hh) {
        f32x4 t[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) t[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        bf16x8 af = take();
        for (int k = 0; k < nk; ++k) {
          bf16x8 an = af;
          if (k + 1 < nk) an = take();
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) t[cb] = mfma16(af, ld_bf16x8(ob + 16 * cb * ols + 32 * k), t[cb]);
          af = an;
        }
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          if (hh == 0 || hu[cb] == hh) uacc[cb] = t[cb];
      }
    }
  }  // latent up-projection
  // the item's partial: per-column maximum m_run (score layout), sum (thread
  // tid < kCols: column tid), output uacc (up-projection layout)
  float l_item = 0.f;
  if (tid < kCols) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) l_item += lred[w * kCols + tid];
  }
  auto store = [&](const f32x4 (&o)[NCB], const float (&m)[2], float l) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const int cl = 16 * (cb0 + cb) + (lane & 15);
      if (cl < cn) {
        const int64_t colg = query_row(c0 + cl, N_g, G, a.H_q);
        *reinterpret_cast<float4*>(a.part_o + (colg * a.n_slots + slot) * D + 16 * ds + 4 * (lane >> 4)) =
            make_float4(o[cb][0], o[cb][1], o[cb][2], o[cb][3]);
      }
    }
    if (tid < cn) {
      const int64_t colg = query_row(c0 + tid, N_g, G, a.H_q);
      a.part_ml[colg * a.n_slots + slot] = make_float2(tid < 32 ? m[0] : m[1], l);
    }
  };
  if constexpr (MAX_RT <= 2) {
    // fold into the group's running partial (log-sum-exp); the group's last
    // item writes it out
    const bool first = (it.flags & kItemFirst) != 0;
    float fa[2], fb[2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      const float mn = first ? m_run[ch] : fmaxf(acc.m[ch], m_run[ch]);
      fa[ch] = first || mn == -INFINITY ? 0.f : fast_exp2(acc.m[ch] - mn);
      fb[ch] = mn == -INFINITY ? 0.f : fast_exp2(m_run[ch] - mn);
      acc.m[ch] = mn;
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const int cc = 16 * (cb0 + cb) + (lane & 15);  // column within the tile
      const bool hi = ((cb0 + cb) >> 1) != 0;        // wave-uniform: column half
      const float sa = __shfl(hi ? fa[1] : fa[0], cc & 31);
      const float sb = __shfl(hi ? fb[1] : fb[0], cc & 31);
      acc.o[cb] = first ? uacc[cb] * sb : acc.o[cb] * sa + uacc[cb] * sb;
    }
    if (tid < kCols) {
      const int ch = tid >> 5;
      acc.l = first ? l_item * fb[ch] : acc.l * fa[ch] + l_item * fb[ch];
    }
    if (it.flags & kItemFlush) store(acc.o, acc.m, acc.l);
  } else {
    store(uacc, m_run, l_item);
  }
}

template <int D, int MAX_RT, int NSLOT, bool WH, int MODE>
__global__ __launch_bounds__(kThreads, 1) void attend_kernel(AttendArgs a) {
  constexpr bool I8 = MODE == 1;
  extern __shared__ __align__(16) unsigned char smem[];
  const WgProgram p = a.wg[blockIdx.x];
  if (p.n_items == 0) return;
  {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(a.prog + p.off);
    uint32_t* dst = reinterpret_cast<uint32_t*>(smem);
    for (int i = threadIdx.x; i < p.words; i += kThreads) dst[i] = src[i];
  }
  lds_barrier();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  unsigned char* work = smem + a.prog_bytes;
  FragRing<D, NSLOT, I8> fr;
  GroupAcc<up_col_blocks<D>()> acc;
  fr.data = reinterpret_cast<const unsigned char*>(a.data);
  fr.lane = threadIdx.x & 63;
  fr.ring = reinterpret_cast<__bf16*>(work + a.ring_offset) + (size_t)wave * NSLOT * kFragElems;
  fr.ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(fr.ring));
  RunDeriver<D> rd;
  rd.items = smem;
  rd.n_items = p.n_items;
  rd.gk = 0;
  rd.gb = 0;
  rd.rbuf = reinterpret_cast<int2*>(smem + (size_t)p.n_items * sizeof(WorkItem));
  rd.recon_delta = a.recon_delta;
  rd.run_cap = a.run_cap;
  fr.run_cap = a.run_cap;
  if (wave == 0) {
    rd.derive(threadIdx.x & 63);
    rd.derive(threadIdx.x & 63);
  }
  lds_barrier();
  fr.rbuf = rd.rbuf + (size_t)wave * kRunBufs * a.run_cap;
  fr.start();
  for (int k = 0; k < p.n_items; ++k) {
    const WorkItem it = lds_item(smem + (size_t)k * sizeof(WorkItem));
    if (k > 0) lds_barrier();  // the previous item's LDS reads are done
    // the thread index is re-derived per item (opaque to the optimiser), so no
    // lane-dependent address of one item kind stays live across the other
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    if (it.kind == kItemBlock) block_item<D, MAX_RT, NSLOT, WH, MODE>(a, it, work, fr, rd, acc, tid);
    else if (it.kind == kItemTail) tail_item<D>(a, it, work, tid);
  }
  if constexpr (NSLOT > 0) wait_vmcnt<0>();  // no LDS write may land after the workgroup ends
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge: one workgroup per query column (i, h).  Its partials are
// the block-group slots [0, nb) of its column tile, then request i's tail
// chunks at n_block_slots + chunk.  Thread t takes the
// 4 output dims 4 (t % (D/4)) of the slots s = t / (D/4) (mod slots per pass),
// so every load is one 16-byte vector and a wave reads whole slots; the loads
// of kMergeUnroll passes are issued before any is used, and each thread keeps
// a running (max, sum, output) over its slots.  The slot lanes are then merged
// in a fixed order through LDS, so the result is deterministic.
// ---------------------------------------------------------------------------
constexpr int kMergeThreads = 256;
constexpr int kMergeUnroll = 8;
template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeArgs a) {
  constexpr int TPS = D / 4;                // threads per slot
  constexpr int SPP = kMergeThreads / TPS;  // slots per pass
  __shared__ float red_m[SPP], red_l[SPP];
  __shared__ float4 red_o[SPP][TPS];
  const int col = blockIdx.x, tid = threadIdx.x;
  const int dq = tid % TPS, sl = tid / TPS;
  const int i = col / a.H_q, h = col % a.H_q;
  const int cf = (h / a.G) * a.tiles.N_g + i * a.G + h % a.G;  // head-major column
  const int nb = a.slot_count[tile_of(a.tiles, cf)];         // block-group slots of its column tile
  const int n_valid = nb + (tail_len_of(a.tl, i) + kTailChunk - 1) / kTailChunk;
  const float2* ml = a.part_ml + (int64_t)col * a.n_slots;
  const float4* po = reinterpret_cast<const float4*>(a.part_o + (int64_t)col * a.n_slots * D) + dq;
  float m = -INFINITY, l = 0.f;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = sl; s0 < n_valid; s0 += SPP * kMergeUnroll) {
    float2 mm[kMergeUnroll];
    float4 oo[kMergeUnroll];
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      const int v = s0 + u * SPP;
      if (v < n_valid) {
        const int s = v < nb ? v : a.n_block_slots + (v - nb);
        mm[u] = ml[s];
        oo[u] = po[(int64_t)s * TPS];
      } else {
        mm[u] = make_float2(-INFINITY, 0.f);
        oo[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      if (mm[u].x == -INFINITY) continue;  // past the last slot
      const float mn = fmaxf(m, mm[u].x);
      const float fo = fast_exp2(m - mn);  // m = -inf before the first slot: 0
      const float fn = fast_exp2(mm[u].x - mn);
      l = l * fo + mm[u].y * fn;
      o.x = o.x * fo + oo[u].x * fn;
      o.y = o.y * fo + oo[u].y * fn;
      o.z = o.z * fo + oo[u].z * fn;
      o.w = o.w * fo + oo[u].w * fn;
      m = mn;
    }
  }
  // every thread of a slot lane holds the same (m, l)
  if (dq == 0) {
    red_m[sl] = m;
    red_l[sl] = l;
  }
  red_o[sl][dq] = o;
  __syncthreads();
  if (tid < TPS) {
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < SPP; ++k) mx = fmaxf(mx, red_m[k]);
    float den = 0.f;
    float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < SPP; ++k) {
      if (red_m[k] == -INFINITY) continue;  // a lane without slots
      const float f = fast_exp2(red_m[k] - mx);
      den += red_l[k] * f;
      const float4 v = red_o[k][tid];
      num.x += v.x * f;
      num.y += v.y * f;
      num.z += v.z * f;
      num.w += v.w * f;
    }
    const float inv = 1.f / den;
    reinterpret_cast<float4*>(a.out + (int64_t)col * D)[tid] =
        make_float4(num.x * inv, num.y * inv, num.z * inv, num.w * inv);
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_pack_batch(const PackArgs* jobs, const int64_t* starts, int n_jobs, int64_t n_frags,
                             hipStream_t s) {
  if (n_jobs == 0 || n_frags == 0) return hipSuccess;
  const int64_t groups = (n_frags + 3) / 4;
  if (groups > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_batch_kernel, dim3((unsigned)groups), dim3(256), 0, s, jobs, starts, n_jobs);
  return hipGetLastError();
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  if (a.n_frags == 0) return hipSuccess;
  const int64_t threads = a.n_frags * 64;
  const unsigned grid = (unsigned)((threads + 255) / 256);
  hipLaunchKernelGGL(pack_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_row_scales(const uint16_t* src, int rows, int cols, int rows_pad, float* scale, int* bad,
                             hipStream_t s) {
  if (rows_pad == 0) return hipSuccess;
  hipLaunchKernelGGL(row_scale_kernel, dim3((rows_pad + 255) / 256), dim3(256), 0, s, src, rows, cols, rows_pad,
                     scale, bad);
  return hipGetLastError();
}

hipError_t launch_scale_units(const float* ks, const float* vs, int T_pad, float* dst, hipStream_t s) {
  if (T_pad == 0) return hipSuccess;
  hipLaunchKernelGGL(scale_units_kernel, dim3((2 * T_pad + 255) / 256), dim3(256), 0, s, ks, vs, T_pad, dst);
  return hipGetLastError();
}


template <int D, int MAX_RT, int NSLOT, bool WH, int MODE>
static hipError_t launch_attend_t(const AttendArgs& a, int grid, size_t lds, hipStream_t s, hipEvent_t e0,
                                  hipEvent_t e1) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_kernel<D, MAX_RT, NSLOT, WH, MODE>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipExtLaunchKernelGGL((attend_kernel<D, MAX_RT, NSLOT, WH, MODE>), dim3(grid), dim3(kThreads), (uint32_t)lds, s,
                        e0, e1, 0, a);
  return hipGetLastError();
}

// ring slots 8 / 6 / none with the whole weight tile; 4 with the half tile
template <int D, int MAX_RT, int MODE>
static hipError_t launch_attend_r(const AttendArgs& a, int nslot, int grid, size_t lds, hipStream_t s, hipEvent_t e0,
                                  hipEvent_t e1) {
  switch (nslot) {
    case 8: return launch_attend_t<D, MAX_RT, 8, false, MODE>(a, grid, lds, s, e0, e1);
    case 6: return launch_attend_t<D, MAX_RT, 6, false, MODE>(a, grid, lds, s, e0, e1);
    case 4: return launch_attend_t<D, MAX_RT, 4, true, MODE>(a, grid, lds, s, e0, e1);
    case 0: return launch_attend_t<D, MAX_RT, 0, false, MODE>(a, grid, lds, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

template <int D, int MODE>
static hipError_t launch_attend_d(const AttendArgs& a, int max_rt, int nslot, int grid, size_t lds,
                                  hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  switch (max_rt) {
    case 2: return launch_attend_r<D, 2, MODE>(a, nslot, grid, lds, s, e0, e1);
    case 3: return launch_attend_r<D, 3, MODE>(a, nslot, grid, lds, s, e0, e1);
    case 4: return launch_attend_r<D, 4, MODE>(a, nslot, grid, lds, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
static hipError_t launch_attend_m(const AttendArgs& a, int max_rt, int nslot, bool p_int8, bool gemv, int grid,
                                  size_t lds, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (p_int8) return launch_attend_d<D, 1>(a, max_rt, nslot, grid, lds, s, e0, e1);
  if (gemv) return launch_attend_d<D, 2>(a, max_rt, nslot, grid, lds, s, e0, e1);
  return launch_attend_d<D, 0>(a, max_rt, nslot, grid, lds, s, e0, e1);
}

hipError_t launch_attend(const AttendArgs& a, int head_dim, int max_rt, int nslot, bool p_int8, bool gemv, int grid,
                         size_t lds_bytes, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (grid == 0) return hipSuccess;
  if (head_dim == 64) return launch_attend_m<64>(a, max_rt, nslot, p_int8, gemv, grid, lds_bytes, s, e0, e1);
  if (head_dim == 128) return launch_attend_m<128>(a, max_rt, nslot, p_int8, gemv, grid, lds_bytes, s, e0, e1);
  return hipErrorInvalidValue;
}

hipError_t launch_merge(const MergeArgs& a, int head_dim, int n_cols, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (head_dim == 64) {
    hipExtLaunchKernelGGL(merge_kernel<64>, dim3(n_cols), dim3(kMergeThreads), 0, s, e0, e1, 0, a);
  } else if (head_dim == 128) {
    hipExtLaunchKernelGGL(merge_kernel<128>, dim3(n_cols), dim3(kMergeThreads), 0, s, e0, e1, 0, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace milo
