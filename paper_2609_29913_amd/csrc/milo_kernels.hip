// gfx950 (CDNA4) kernels for decode attention over a block-wise low-rank KV
// cache (MILO, Sec. 4.2 Eq. 3 factors; Sec. 4.4 Alg. 1 inference stage; the
// attention itself is Sec. 4.1 Eq. 1).
//
//  pack_kernel    repacks row-major bf16 factors into MFMA-fragment order.
//  attend_kernel  persistent: one workgroup per compute unit runs a host-built
//                 list of work items, its fragment streams flowing across items:
//     block item (block b, KV head g, 64-column tile of query columns):
//       projection  Qt = scale*log2(e) * R^K_b[:, g] q          (MFMA, into LDS)
//       scores      S  = P^K_b Qt, 256 tokens per tile          (MFMA, 4 waves x 64 tokens)
//       softmax     running max per column shared by the waves, W = 2^(S - m)
//       latent V    Ot = sum_t W_t P^V_b[t]                      (MFMA, waves split the rank)
//       up-project  o  = R^V_b[:, g]^T Ot                        (MFMA from registers)
//       -> partial (m, l, o) per column
//     tail item (request i, KV head g, 128-token chunk of the request's own KV):
//       plain attention of the group's query heads over the chunk (VALU, LDS-staged)
//       -> partial (m, l, o) per column
//  merge_kernel   log-sum-exp merge of every partial of a column into O (fp32).
//
// Scores are kept in log2 units (the scale folds log2(e)), so every exponential
// is one v_exp_f32.
#include "milo_internal.h"

namespace milo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8 ld_bf16x8(const void* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ void lds_dma16(const uint16_t* g, __bf16* lds_slot) {
  __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(g),
                                   reinterpret_cast<__attribute__((address_space(3))) void*>(
                                       reinterpret_cast<uintptr_t>(lds_slot)),
                                   16, 0, 0);
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

// Workgroup barrier for the attention kernel: every wave's LDS reads and
// writes issued before it are complete.  In-flight global->LDS fragment loads
// are deliberately not waited for (each targets its own wave's ring slots);
// __syncthreads() would make the compiler drain them (vmcnt(0)) at many
// barriers.  The "memory" clobber keeps the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0xF70 | N);  // vmcnt(N), expcnt/lgkmcnt not waited
}

// ---------------------------------------------------------------------------
// Packing
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_kernel(PackArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t frag = gid >> 6;
  const int lane = (int)(gid & 63);
  if (frag >= a.n_frags) return;
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

// ---------------------------------------------------------------------------
// Tail work item: attention of the G query heads of KV head g of request i over
// tokens [t0, t0 + nt) of that request's uncompressed KV (nt <= 128 comes with
// the item).  Wave w takes tokens t0 + 32w .. t0 + 32w + 31; every load of the
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
  const int i = it.req, slot = it.slot, g = it.g, G = a.G;
  const int wave = tid >> 6, lane = tid & 63, lrow = lane & 31, lhi = lane >> 5;
  const int t0 = it.sub * kTailChunk, nt = it.blk.T;
  float* red = reinterpret_cast<float*>(smem);   // [kWaves][32] column maxima
  float* lred = red + kWaves * 32;               // [kWaves][32] column sums
  float* wt = lred + kWaves * 32;                // [kTailChunk][32] weights, token-major
  float* op = wt + kTailChunk * 32;              // [kWaves][kMaxGroup][D] partial outputs

  const int64_t rs = (int64_t)a.H_kv * D;      // row stride of the tail K / V
  const int64_t row0 = (int64_t)i * a.tail_cap + t0;
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

// ---------------------------------------------------------------------------
// Block work item: latent-space attention of one 64-column tile of the query
// columns of KV head g over the tiles [tile0, tile0 + ntile) of block b.
//
// Waves split the tokens of each 256-token tile for the scores (64 tokens each)
// and split the rank tiles of the latent accumulator (rank tile rt belongs to
// wave rt % 4).  Every factor fragment a wave consumes (R^K for the projection,
// P^K and P^V per tile, R^V for the up-projection) comes from the wave's
// fragment stream (FragRing below).  Every loop is software-pipelined: the
// operands of step k+1 are read while the MFMAs of step k run.
// ---------------------------------------------------------------------------
// A wave's fragment stream over all block items of its workgroup.  The host
// lists, per wave, the runs of consecutive packed fragments in the order the
// wave consumes them (per block item: its R^K run for the projection, then for
// every 256-token tile its P^K run and its P^V run, then its R^V run for the
// up-projection); the list sits in LDS and ends with a long sentinel run.
// With NSLOT > 0 fragments reach the wave through a private ring of NSLOT LDS
// slots, filled by direct global->LDS loads issued kDepth fragments ahead of
// use, so every wait is a constant vmcnt; the look-ahead crosses item
// boundaries, so the next item's first fragments load while the current one
// finishes.  With NSLOT == 0 fragments are loaded straight into registers.
// All fields are wave-uniform (scalar registers).
template <int NSLOT>
struct FragRing {
  static constexpr int kDepth = NSLOT > 2 ? NSLOT - 2 : 1;  // fragments in flight
  const uint16_t* data_lane;  // packed buffer + this lane's 8-element offset
  __bf16* ring;               // this wave's NSLOT slots
  const int2* run;            // current entry of this wave's run list (LDS)
  int64_t off;                // element offset of the next fragment
  int left;                   // fragments left in the current run
  int rs, ws;                 // ring slots: next to read, next to fill
  int lane8;                  // this lane's element offset inside a fragment

  __device__ __forceinline__ void load_run() {
    const int2 v = prog_read_b64(run);
    off = (int64_t)__builtin_amdgcn_readfirstlane(v.x) * kFragElems;
    left = __builtin_amdgcn_readfirstlane(v.y);
  }
  // offset of the next fragment of the stream; advances it
  __device__ __forceinline__ int64_t next() {
    const int64_t o = off;
    off += kFragElems;
    if (--left == 0) {
      ++run;
      load_run();
    }
    return o;
  }
  __device__ __forceinline__ void start() {
    load_run();
    rs = 0;
    ws = 0;
    if constexpr (NSLOT > 0) {
#pragma unroll
      for (int k = 0; k < kDepth; ++k) lds_dma16(data_lane + next(), ring + k * kFragElems);
      ws = kDepth;
    }
  }
  // the next fragment, in this lane's operand layout
  __device__ __forceinline__ bf16x8 take() {
    if constexpr (NSLOT > 0) {
      wait_vmcnt<kDepth - 1>();
      const bf16x8 v = ld_bf16x8(ring + rs * kFragElems + lane8);
      lds_dma16(data_lane + next(), ring + ws * kFragElems);
      rs = rs + 1 == NSLOT ? 0 : rs + 1;
      ws = ws + 1 == NSLOT ? 0 : ws + 1;
      return v;
    } else {
      return ld_bf16x8(data_lane + next());
    }
  }
};

template <int D, int MAX_RT, int NSLOT>
__device__ __forceinline__ void block_item(const AttendArgs& a, const WorkItem& it, unsigned char* smem,
                                           FragRing<NSLOT>& fr, const int tid) {
  constexpr int NK = D / 16;
  const BlockMeta& bm = it.blk;
  const int slot = it.slot, g = it.g, c0 = it.sub * kCols;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 31, lhi = lane >> 5;
  const int G = a.G, ncg = a.n_q * G;
  const int qsd = a.qt_stride;
  const int nrt_k = bm.rk_pad >> 5, nks = bm.rk_pad >> 4;
  const int nrt_v = bm.rv_pad >> 5, nkv = bm.rv_pad >> 4;
  const int my_nrt = owned_tiles(nrt_v, wave);
  const int my_nrt_k = owned_tiles(nrt_k, wave);
  const int T = bm.T;
  const int ntiles = it.ntile, tile0 = it.tile0;  // tiles this item covers
  __bf16* qt = reinterpret_cast<__bf16*>(smem);              // [kCols][qsd]
  __bf16* wl = qt + kCols * qsd;                               // [kCols][kWStride]
  float* red = reinterpret_cast<float*>(wl + kCols * kWStride);  // [kWaves][kCols]
  // the wave's next fragment; the order of take() calls below is the order of
  // the wave's runs: R^K, then per tile P^K and P^V, then R^V
  auto take = [&]() -> bf16x8 { return fr.take(); };

  // ---- projection: Qt[rank][col] (stored [col][rank]) ----
  {
    bf16x8 qf[NK][2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      const int c = c0 + 32 * ch + lrow;
      const bool ok = c < ncg;
      const int qi = ok ? c / G : 0, qh = ok ? g * G + c % G : 0;
      const uint16_t* qrow = a.q + ((int64_t)qi * a.H_q + qh) * D + 8 * lhi;
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        bf16x8 v = ld_bf16x8(qrow + 16 * k);
        qf[k][ch] = ok ? v : bf16x8{};
      }
    }
    for (int j = 0; j < my_nrt_k; ++j) {
      const int rt = wave + kWaves * j;
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
        *reinterpret_cast<bf16x4*>(qt + lrow * qsd + r) = v0;
        *reinterpret_cast<bf16x4*>(qt + (32 + lrow) * qsd + r) = v1;
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
  const __bf16* qr0 = qt + lrow * qsd + 8 * lhi;
  const __bf16* qr1 = qt + (32 + lrow) * qsd + 8 * lhi;
  const __bf16* wr0 = wl + lrow * kWStride + 8 * lhi;
  const __bf16* wr1 = wl + (32 + lrow) * kWStride + 8 * lhi;

  for (int tt = 0; tt < ntiles; ++tt) {
    const int t0 = (tile0 + tt) * kTile;
    const int tw = t0 + wave * kTokWave;
    f32x16 s00 = {}, s01 = {}, s10 = {}, s11 = {};
    {
      // operands of rank step k: a0/a1 (P^K sub-tiles), b0/b1 (Qt column tiles);
      // nks is even (ranks are padded to 32), so the loop runs over step pairs
      bf16x8 a0 = take(), a1 = take();
      bf16x8 b0 = ld_bf16x8(qr0), b1 = ld_bf16x8(qr1);
      for (int k = 0; k < nks; k += 2) {
        const bf16x8 c0 = take(), c1 = take();
        const bf16x8 d0 = ld_bf16x8(qr0 + 16 * (k + 1));
        const bf16x8 d1 = ld_bf16x8(qr1 + 16 * (k + 1));
        s00 = mfma32(a0, b0, s00);
        s01 = mfma32(a0, b1, s01);
        s10 = mfma32(a1, b0, s10);
        s11 = mfma32(a1, b1, s11);
        if (k + 2 < nks) {
          a0 = take();
          a1 = take();
          b0 = ld_bf16x8(qr0 + 16 * (k + 2));
          b1 = ld_bf16x8(qr1 + 16 * (k + 2));
        }
        s00 = mfma32(c0, d0, s00);
        s01 = mfma32(c0, d1, s01);
        s10 = mfma32(c1, d0, s10);
        s11 = mfma32(c1, d1, s11);
      }
    }
    f32x16 s[2][2] = {{s00, s01}, {s10, s11}};
    // mask tokens past the end of the block, wave-local column max
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int tok = tw + 32 * mt + 8 * (v >> 2) + 4 * lhi + (v & 3);
          const float x = tok < T ? s[mt][ch][v] : -INFINITY;
          s[mt][ch][v] = x;
          mx[ch] = fmaxf(mx[ch], x);
        }
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      mx[ch] = fmaxf(mx[ch], __shfl_xor(mx[ch], 32));
      if (lhi == 0) red[wave * kCols + 32 * ch + lrow] = mx[ch];
    }
    lds_barrier();
    float alpha[2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      float tm = red[32 * ch + lrow];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) tm = fmaxf(tm, red[w * kCols + 32 * ch + lrow]);
      const float mn = fmaxf(m_run[ch], tm);
      alpha[ch] = fast_exp2(m_run[ch] - mn);
      m_run[ch] = mn;
    }
    // weights -> LDS as [col][token] bf16
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      float lsum = 0.f;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bf16x4 w4;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float w = fast_exp2(s[mt][ch][4 * j + u] - m_run[ch]);
            lsum += w;
            w4[u] = (__bf16)w;
          }
          *reinterpret_cast<bf16x4*>(wl + (32 * ch + lrow) * kWStride + wave * kTokWave + 32 * mt +
                                     8 * j + 4 * lhi) = w4;
        }
      l_run[ch] = l_run[ch] * alpha[ch] + lsum;
    }
    lds_barrier();
#pragma unroll
    for (int r = 0; r < MAX_RT; ++r) {
      oacc[r][0] *= alpha[0];
      oacc[r][1] *= alpha[1];
    }
    if (my_nrt > 0) {
      // operands of 16-token step sg: w0/w1 (weight column tiles), pa[r] (P^V rank tiles)
      bf16x8 pa[MAX_RT], pc[MAX_RT];
      bf16x8 w0 = ld_bf16x8(wr0), w1 = ld_bf16x8(wr1);
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r)
        if (r < my_nrt) pa[r] = take();
      for (int sg = 0; sg < kTile / 16; sg += 2) {
        const bf16x8 x0 = ld_bf16x8(wr0 + 16 * (sg + 1));
        const bf16x8 x1 = ld_bf16x8(wr1 + 16 * (sg + 1));
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < my_nrt) pc[r] = take();
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < my_nrt) {
            oacc[r][0] = mfma32(pa[r], w0, oacc[r][0]);
            oacc[r][1] = mfma32(pa[r], w1, oacc[r][1]);
          }
        if (sg + 2 < kTile / 16) {
          w0 = ld_bf16x8(wr0 + 16 * (sg + 2));
          w1 = ld_bf16x8(wr1 + 16 * (sg + 2));
#pragma unroll
          for (int r = 0; r < MAX_RT; ++r)
            if (r < my_nrt) pa[r] = take();
        }
#pragma unroll
        for (int r = 0; r < MAX_RT; ++r)
          if (r < my_nrt) {
            oacc[r][0] = mfma32(pc[r], x0, oacc[r][0]);
            oacc[r][1] = mfma32(pc[r], x1, oacc[r][1]);
          }
      }
    }
  }

  // ---- up-projection through R^V and the partial (m, l, o) ----
#pragma unroll
  for (int ch = 0; ch < 2; ++ch) l_run[ch] += __shfl_xor(l_run[ch], 32);
  lds_barrier();  // every wave is done with qt / wl
  float* ored = reinterpret_cast<float*>(smem);       // [kWaves][kCols][kORow]
  float* lred = ored + kWaves * kCols * kORow;        // [kWaves][kCols]
  if (lhi == 0) {
    lred[wave * kCols + lrow] = l_run[0];
    lred[wave * kCols + 32 + lrow] = l_run[1];
  }
#pragma unroll
  for (int pass = 0; pass < D / 64; ++pass) {
    f32x16 acc[2][2];
    acc[0][0] = acc[0][1] = acc[1][0] = acc[1][1] = f32x16{};
    if (my_nrt > 0) {
      // fragments of (owned rank tile r, rank half, d tile dt), in stream order
      bf16x8 f00 = take(), f01 = take();
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r) {
        if (r < my_nrt) {
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            // prefetch the next (rank tile, half) pair of d-tile fragments
            bf16x8 g00 = f00, g01 = f01;
            if (half == 0 || r + 1 < my_nrt) {
              g00 = take();
              g01 = take();
            }
            bf16x8 b0, b1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              b0[e] = (__bf16)oacc[r][0][8 * half + e];
              b1[e] = (__bf16)oacc[r][1][8 * half + e];
            }
            acc[0][0] = mfma32(f00, b0, acc[0][0]);
            acc[0][1] = mfma32(f00, b1, acc[0][1]);
            acc[1][0] = mfma32(f01, b0, acc[1][0]);
            acc[1][1] = mfma32(f01, b1, acc[1][1]);
            f00 = g00;
            f01 = g01;
          }
        }
      }
    }
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float4 v = make_float4(acc[dt][ch][4 * j], acc[dt][ch][4 * j + 1], acc[dt][ch][4 * j + 2],
                                 acc[dt][ch][4 * j + 3]);
          *reinterpret_cast<float4*>(ored + (wave * kCols + 32 * ch + lrow) * kORow + 32 * dt + 8 * j +
                                     4 * lhi) = v;
        }
    lds_barrier();
    {
      const int col = tid >> 2, dq = (tid & 3) * 16;
      const int c = c0 + col;
      if (c < ncg) {
        const int64_t colg = (int64_t)(c / G) * a.H_q + g * G + c % G;
        float* dst = a.part_o + (colg * a.n_slots + slot) * D + 64 * pass + dq;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float4 sum = *reinterpret_cast<const float4*>(ored + col * kORow + dq + 4 * q4);
#pragma unroll
          for (int w = 1; w < kWaves; ++w) {
            const float4 x = *reinterpret_cast<const float4*>(ored + (w * kCols + col) * kORow + dq + 4 * q4);
            sum.x += x.x; sum.y += x.y; sum.z += x.z; sum.w += x.w;
          }
          *reinterpret_cast<float4*>(dst + 4 * q4) = sum;
        }
      }
    }
    lds_barrier();
  }
  if (tid < kCols) {
    const int c = c0 + tid;
    if (c < ncg) {
      float l = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) l += lred[w * kCols + tid];
      const float m = tid < 32 ? m_run[0] : m_run[1];
      const int64_t colg = (int64_t)(c / G) * a.H_q + g * G + c % G;
      a.part_ml[colg * a.n_slots + slot] = make_float2(m, l);
    }
  }
}

// a work item read from LDS into wave-uniform registers
__device__ __forceinline__ WorkItem lds_item(const unsigned char* p) {
  static_assert(sizeof(WorkItem) % 16 == 0, "work items are whole 16-byte chunks");
  int32_t w[sizeof(WorkItem) / 4];
#pragma unroll
  for (int i = 0; i < (int)sizeof(WorkItem) / 16; ++i) {
    const int4 v = prog_read_b128(p + 16 * i);
    w[4 * i + 0] = __builtin_amdgcn_readfirstlane(v.x);
    w[4 * i + 1] = __builtin_amdgcn_readfirstlane(v.y);
    w[4 * i + 2] = __builtin_amdgcn_readfirstlane(v.z);
    w[4 * i + 3] = __builtin_amdgcn_readfirstlane(v.w);
  }
  WorkItem it;
  __builtin_memcpy(&it, w, sizeof(WorkItem));
  return it;
}

template <int D, int MAX_RT, int NSLOT>
__global__ __launch_bounds__(kThreads, 1) void attend_kernel(AttendArgs a) {
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
  const int run_off = wave == 0 ? p.run_off[0] : wave == 1 ? p.run_off[1] : wave == 2 ? p.run_off[2] : p.run_off[3];
  unsigned char* work = smem + a.prog_bytes;
  FragRing<NSLOT> fr;
  fr.data_lane = a.data + (threadIdx.x & 63) * 8;
  fr.lane8 = (threadIdx.x & 63) * 8;
  fr.run = reinterpret_cast<const int2*>(smem + run_off);
  fr.ring = reinterpret_cast<__bf16*>(work + a.ring_offset) + (size_t)wave * NSLOT * kFragElems;
  fr.start();
  for (int k = 0; k < p.n_items; ++k) {
    const WorkItem it = lds_item(smem + (size_t)k * sizeof(WorkItem));
    if (k > 0) lds_barrier();  // the previous item's LDS reads are done
    // the thread index is re-derived per item (opaque to the optimiser), so no
    // lane-dependent address of one item kind stays live across the other
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    if (it.kind == kItemBlock) block_item<D, MAX_RT, NSLOT>(a, it, work, fr, tid);
    else if (it.kind == kItemTail) tail_item<D>(a, it, work, tid);
  }
  if constexpr (NSLOT > 0) wait_vmcnt<0>();  // no LDS write may land after the workgroup ends
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge: one workgroup per query column (i, h).  Slots [0, n_sel)
// are the selected blocks, then request i's tail chunks.  Wave w accumulates
// the slots s = w mod 4 (each lane owns D/64 consecutive outputs); the waves are
// combined in a fixed order, so the result is deterministic.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void merge_kernel(MergeArgs a) {
  constexpr int E = D / 64;  // outputs per lane
  __shared__ float red[kWaves];
  __shared__ float dred[kWaves];
  __shared__ float part[kWaves][D];
  const int col = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i = col / a.H_q;
  const int n_valid = a.n_block_slots + (a.tail_len[i] + kTailChunk - 1) / kTailChunk;
  const float2* ml = a.part_ml + (int64_t)col * a.n_slots;
  float mx = -INFINITY;
  for (int s = tid; s < n_valid; s += kThreads) mx = fmaxf(mx, ml[s].x);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float num[E], den = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) num[e] = 0.f;
  const float* po = a.part_o + (int64_t)col * a.n_slots * D + E * lane;
  int s = wave;
  for (; s + 3 * kWaves < n_valid; s += 4 * kWaves) {
    float2 m4[4];
    float v4[4][E];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      m4[u] = ml[s + u * kWaves];
#pragma unroll
      for (int e = 0; e < E; ++e) v4[u][e] = po[(int64_t)(s + u * kWaves) * D + e];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float f = fast_exp2(m4[u].x - mx);
      den += m4[u].y * f;
#pragma unroll
      for (int e = 0; e < E; ++e) num[e] += v4[u][e] * f;
    }
  }
  for (; s < n_valid; s += kWaves) {
    const float2 m1 = ml[s];
    const float f = fast_exp2(m1.x - mx);
    den += m1.y * f;
#pragma unroll
    for (int e = 0; e < E; ++e) num[e] += po[(int64_t)s * D + e] * f;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) part[wave][E * lane + e] = num[e];
  if (lane == 0) dred[wave] = den;
  __syncthreads();
  if (tid < D) {
    const float dsum = dred[0] + dred[1] + dred[2] + dred[3];
    const float nsum = part[0][tid] + part[1][tid] + part[2][tid] + part[3][tid];
    a.out[(int64_t)col * D + tid] = nsum / dsum;
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  if (a.n_frags == 0) return hipSuccess;
  const int64_t threads = a.n_frags * 64;
  const unsigned grid = (unsigned)((threads + 255) / 256);
  hipLaunchKernelGGL(pack_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

size_t attend_lds_base_bytes(int head_dim, int rk_pad_max) {
  const size_t qsd = (size_t)rk_pad_max + 8;
  const size_t loop = kCols * qsd * 2 + (size_t)kCols * kWStride * 2 + (size_t)kWaves * kCols * 4;
  const size_t epi = ((size_t)kWaves * kCols * kORow + (size_t)kWaves * kCols) * 4;
  const size_t tail = ((size_t)2 * kWaves * 32 + (size_t)kTailChunk * 32 + (size_t)kWaves * kMaxGroup * head_dim) * 4;
  size_t m = loop > epi ? loop : epi;
  m = m > tail ? m : tail;
  return (m + 1023) / 1024 * 1024;  // the fragment rings start here
}

size_t attend_ring_bytes(int nslot) { return (size_t)kWaves * nslot * kFragElems * 2; }

template <int D, int MAX_RT, int NSLOT>
static hipError_t launch_attend_t(const AttendArgs& a, int grid, size_t lds, hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_kernel<D, MAX_RT, NSLOT>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((attend_kernel<D, MAX_RT, NSLOT>), dim3(grid), dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

template <int D, int MAX_RT>
static hipError_t launch_attend_r(const AttendArgs& a, int nslot, int grid, size_t lds, hipStream_t s) {
  switch (nslot) {
    case 14: return launch_attend_t<D, MAX_RT, 14>(a, grid, lds, s);
    case 12: return launch_attend_t<D, MAX_RT, 12>(a, grid, lds, s);
    case 6: return launch_attend_t<D, MAX_RT, 6>(a, grid, lds, s);
    case 0: return launch_attend_t<D, MAX_RT, 0>(a, grid, lds, s);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
static hipError_t launch_attend_d(const AttendArgs& a, int max_rt, int nslot, int grid, size_t lds,
                                  hipStream_t s) {
  switch (max_rt) {
    case 2: return launch_attend_r<D, 2>(a, nslot, grid, lds, s);
    case 4: return launch_attend_r<D, 4>(a, nslot, grid, lds, s);
    case 6: return launch_attend_r<D, 6>(a, nslot, grid, lds, s);
    case 8: return launch_attend_r<D, 8>(a, nslot, grid, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attend(const AttendArgs& a, int head_dim, int max_rt, int nslot, int grid, size_t lds_bytes,
                         hipStream_t s) {
  if (grid == 0) return hipSuccess;
  if (head_dim == 64) return launch_attend_d<64>(a, max_rt, nslot, grid, lds_bytes, s);
  if (head_dim == 128) return launch_attend_d<128>(a, max_rt, nslot, grid, lds_bytes, s);
  return hipErrorInvalidValue;
}

hipError_t launch_merge(const MergeArgs& a, int head_dim, int n_cols, hipStream_t s) {
  if (head_dim == 64) {
    hipLaunchKernelGGL(merge_kernel<64>, dim3(n_cols), dim3(kThreads), 0, s, a);
  } else if (head_dim == 128) {
    hipLaunchKernelGGL(merge_kernel<128>, dim3(n_cols), dim3(kThreads), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace milo
