// gfx950 (CDNA4) kernels for decode attention over a block-wise low-rank KV
// cache (MILO, Sec. 4.2 Eq. 3 factors; Sec. 4.4 Alg. 1 inference stage; the
// attention itself is Sec. 4.1 Eq. 1).
//
//  pack_kernel    repacks row-major bf16 factors into MFMA-fragment order.
//  attend_kernel  one workgroup per work item:
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
// tokens [t0, t0 + nt) of that request's uncompressed KV.  The chunk's K and V
// rows are staged in LDS with coalesced 16-byte loads, then scored and
// accumulated from LDS.
// ---------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ void tail_item(const AttendArgs& a, const WorkItem& it, unsigned char* smem) {
  constexpr int kRow = D + 8;               // bf16 row stride of the staged K / V
  constexpr int kChunks = D / 8;            // 16-byte pieces per row
  constexpr int kPairs = D / 2;             // d pairs of the value pass (one per lane)
  const int i = it.req, slot = it.slot, g = it.g;
  const int G = a.G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int t0 = it.sub * kTailChunk;
  const int nt = min(kTailChunk, a.tail_len[i] - t0);
  __bf16* kt = reinterpret_cast<__bf16*>(smem);           // [kTailChunk][kRow]
  __bf16* vt = kt + kTailChunk * kRow;                      // [kTailChunk][kRow]
  float* qs = reinterpret_cast<float*>(vt + kTailChunk * kRow);  // [kMaxGroup][D]
  float* sc = qs + kMaxGroup * D;                           // [kTailChunk][kMaxGroup] token-major
  float2* ml = reinterpret_cast<float2*>(sc + kMaxGroup * kTailChunk);  // [kMaxGroup]
  float* op = reinterpret_cast<float*>(kt);  // [kWaves][kMaxGroup][D], over K (dead after scoring)

  const int64_t rstride = (int64_t)a.H_kv * D;
  const uint16_t* kb = a.tail_k + ((int64_t)i * a.tail_cap + t0) * rstride + (int64_t)g * D;
  const uint16_t* vb = a.tail_v + ((int64_t)i * a.tail_cap + t0) * rstride + (int64_t)g * D;
  {
    // every load of the chunk is issued before the first LDS write; rows past
    // the chunk's end re-read its last row (never used), so no load is predicated
    constexpr int kPer = kTailChunk * kChunks / kThreads;
    constexpr int kQPer = kMaxGroup * D / kThreads;
    uint4 kv[kPer], vv[kPer];
    uint16_t qv[kQPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int x = tid + u * kThreads, t = min(x / kChunks, nt - 1), c = x % kChunks;
      kv[u] = *reinterpret_cast<const uint4*>(kb + t * rstride + 8 * c);
      vv[u] = *reinterpret_cast<const uint4*>(vb + t * rstride + 8 * c);
    }
#pragma unroll
    for (int u = 0; u < kQPer; ++u) {
      const int x = tid + u * kThreads, hh = min(x / D, G - 1), j = x % D;
      qv[u] = a.q[((int64_t)i * a.H_q + g * G + hh) * D + j];
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int x = tid + u * kThreads, t = x / kChunks, c = x % kChunks;
      *reinterpret_cast<uint4*>(kt + t * kRow + 8 * c) = kv[u];
      *reinterpret_cast<uint4*>(vt + t * kRow + 8 * c) = vv[u];
    }
#pragma unroll
    for (int u = 0; u < kQPer; ++u) qs[tid + u * kThreads] = bf16_to_f32(qv[u]) * a.qscale;
  }
  __syncthreads();
  // scores: thread (token t, head parity hp) covers heads hp, hp+2, ...; the
  // loops run over the largest group size without branches (heads past G read
  // the last head's query and are discarded), so the LDS reads pipeline
  {
    const int t = tid % kTailChunk, hp = tid / kTailChunk;
    float acc[kMaxGroup / 2];
#pragma unroll
    for (int u = 0; u < kMaxGroup / 2; ++u) acc[u] = 0.f;
    const __bf16* kr = kt + t * kRow;
    const float* qh[kMaxGroup / 2];
#pragma unroll
    for (int u = 0; u < kMaxGroup / 2; ++u) qh[u] = qs + min(hp + 2 * u, G - 1) * D;
#pragma unroll 2
    for (int j = 0; j < D; j += 8) {
      const bf16x8 k8 = ld_bf16x8(kr + j);
      float kf[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) kf[e] = (float)k8[e];
#pragma unroll
      for (int u = 0; u < kMaxGroup / 2; ++u) {
        const float4 qa = *reinterpret_cast<const float4*>(qh[u] + j);
        const float4 qb = *reinterpret_cast<const float4*>(qh[u] + j + 4);
        acc[u] += kf[0] * qa.x + kf[1] * qa.y + kf[2] * qa.z + kf[3] * qa.w +
                  kf[4] * qb.x + kf[5] * qb.y + kf[6] * qb.z + kf[7] * qb.w;
      }
    }
    if (t < nt) {
#pragma unroll
      for (int u = 0; u < kMaxGroup / 2; ++u) {
        const int hh = hp + 2 * u;
        if (hh < G) sc[t * kMaxGroup + hh] = acc[u];
      }
    }
  }
  __syncthreads();
  for (int hh = wave; hh < G; hh += kWaves) {
    float mx = -INFINITY;
    for (int t = lane; t < nt; t += 64) mx = fmaxf(mx, sc[t * kMaxGroup + hh]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.f;
    for (int t = lane; t < nt; t += 64) {
      const float w = fast_exp2(sc[t * kMaxGroup + hh] - mx);
      sc[t * kMaxGroup + hh] = w;
      sum += w;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) ml[hh] = make_float2(mx, sum);
  }
  __syncthreads();
  // values: lane owns the d pair (2*dp, 2*dp+1) for D == 128 (one d for D == 64),
  // wave w the tokens w, w+4, ...; every head of the group at once
  {
    constexpr int kDL = D / 64;  // d values per lane
    float acc[kMaxGroup][kDL];
#pragma unroll
    for (int hh = 0; hh < kMaxGroup; ++hh)
#pragma unroll
      for (int e = 0; e < kDL; ++e) acc[hh][e] = 0.f;
    const int d0 = kDL * lane;
#pragma unroll 4
    for (int t = wave; t < nt; t += kWaves) {
      float v[kDL];
#pragma unroll
      for (int e = 0; e < kDL; ++e) v[e] = (float)vt[t * kRow + d0 + e];
      const float4* wr = reinterpret_cast<const float4*>(sc + t * kMaxGroup);
#pragma unroll
      for (int q4 = 0; q4 < kMaxGroup / 4; ++q4) {
        const float4 w4 = wr[q4];  // weights past G are unset and their sums discarded
        const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int e = 0; e < kDL; ++e) acc[4 * q4 + u][e] += wv[u] * v[e];
      }
    }
#pragma unroll
    for (int hh = 0; hh < kMaxGroup; ++hh)
      if (hh < G)
#pragma unroll
        for (int e = 0; e < kDL; ++e) op[(wave * kMaxGroup + hh) * D + d0 + e] = acc[hh][e];
  }
  __syncthreads();
  for (int x = tid; x < G * D; x += kThreads) {
    const int hh = x / D, jj = x % D;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += op[(w * kMaxGroup + hh) * D + jj];
    const int64_t col = (int64_t)i * a.H_q + g * G + hh;
    a.part_o[(col * a.n_slots + slot) * D + jj] = s;
    if (jj == 0) a.part_ml[col * a.n_slots + slot] = ml[hh];
  }
}

// ---------------------------------------------------------------------------
// Block work item: latent-space attention of one 64-column tile of the query
// columns of KV head g over all tokens of block b.
//
// Waves split the tokens of each 256-token tile for the scores (64 tokens each)
// and split the rank tiles of the latent accumulator (rank tile rt belongs to
// wave rt % 4).  Every factor fragment a wave consumes (R^K for the projection,
// P^K and P^V per tile, R^V for the up-projection) forms one stream per work
// item.  With NSLOT > 0 the stream is fed through a private ring of NSLOT LDS
// slots by direct global->LDS loads issued kDepth fragments ahead of use (so
// each wait is a constant vmcnt); with NSLOT == 0 fragments are loaded
// straight into registers.  Every loop is software-pipelined: the operands of
// step k+1 are read while the MFMAs of step k run.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lds_dma16(const uint16_t* g, __bf16* lds_slot) {
  __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(g),
                                   reinterpret_cast<__attribute__((address_space(3))) void*>(
                                       reinterpret_cast<uintptr_t>(lds_slot)),
                                   16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0xF70 | N);  // vmcnt(N), expcnt/lgkmcnt not waited
}

// A wave's fragment stream.  In consumption order it is: the wave's R^K run
// (projection), then for every 256-token tile the next 2*nks fragments of its
// P^K run and the next 16*my_nrt fragments of its P^V run, then its R^V run
// (up-projection).  The packed layout stores each of these runs contiguously,
// so advancing is an add and a countdown; the phase changes only when a run
// ends.  Once exhausted, the stream keeps returning its last fragment.  All
// fields are wave-uniform (scalar registers).
struct FragStream {
  int64_t off;        // element offset of the next fragment
  int64_t step;       // kFragElems while running, 0 once exhausted
  int left;           // fragments left in the current run
  int phase, t;       // 0 R^K, 1 P^K of tile t, 2 P^V of tile t, 3 R^V, 4 exhausted
  int64_t pk, pv, rv; // resume points of the wave's P^K / P^V runs, start of its R^V run
  int n_pk, n_pv, n_rv, ntiles;

  __device__ __forceinline__ void begin_tile() {
    phase = 1;
    off = pk;
    left = n_pk;
  }
  __device__ __forceinline__ void finish() {
    phase = 4;
    off -= kFragElems;
    step = 0;
    left = 1 << 30;
  }
  __device__ __forceinline__ void init(int64_t rk, int n_rk) {
    t = 0;
    step = kFragElems;
    if (n_rk > 0) {
      phase = 0;
      off = rk;
      left = n_rk;
    } else {
      begin_tile();
    }
  }
  __device__ void next_tile() {
    if (++t < ntiles) {
      begin_tile();
    } else if (n_rv > 0) {
      phase = 3;
      off = rv;
      left = n_rv;
    } else {
      finish();
    }
  }
  __device__ void refill() {
    switch (phase) {
      case 0: begin_tile(); break;
      case 1:
        pk = off;
        if (n_pv > 0) {
          phase = 2;
          off = pv;
          left = n_pv;
        } else {
          next_tile();
        }
        break;
      case 2: pv = off; next_tile(); break;
      default: finish(); break;  // end of the R^V run
    }
  }
  // offset of the next fragment; advances the stream
  __device__ __forceinline__ int64_t next() {
    const int64_t o = off;
    off += step;
    if (--left == 0) refill();
    return o;
  }
};

template <int D, int MAX_RT, int NSLOT>
__device__ __forceinline__ void block_item(const AttendArgs& a, const WorkItem& it, unsigned char* smem) {
  constexpr int kDepth = NSLOT > 2 ? NSLOT - 2 : 1;   // fragments in flight per wave
  constexpr int NK = D / 16;
  const BlockMeta& bm = it.blk;
  const int slot = it.slot, g = it.g, c0 = it.sub * kCols;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 31, lhi = lane >> 5;
  const int G = a.G, ncg = a.n_q * G;
  const int qsd = a.qt_stride;
  const int nrt_k = bm.rk_pad >> 5, nks = bm.rk_pad >> 4;
  const int nrt_v = bm.rv_pad >> 5, nkv = bm.rv_pad >> 4;
  const int my_nrt = owned_tiles(nrt_v, wave);
  const int my_nrt_k = owned_tiles(nrt_k, wave);
  const int T = bm.T;
  const int tiles_all = bm.T_pad / kTile;     // tiles of the whole block (run lengths)
  const int ntiles = it.ntile, tile0 = it.tile0;  // tiles this item covers
  __bf16* qt = reinterpret_cast<__bf16*>(smem);              // [kCols][qsd]
  __bf16* wl = qt + kCols * qsd;                               // [kCols][kWStride]
  float* red = reinterpret_cast<float*>(wl + kCols * kWStride);  // [kWaves][kCols]
  const uint16_t* data_lane = a.data + lane * 8;

  // ---- start streaming fragments before anything else ----
  FragStream st;
  st.pk = bm.off_pk + ((int64_t)wave * tiles_all + tile0) * 2 * nks * kFragElems;
  st.pv = bm.off_pv + ((int64_t)(bm.T_pad / 16) * owned_before(nrt_v, wave) + (int64_t)tile0 * 16 * my_nrt) * kFragElems;
  st.rv = bm.off_rv + ((int64_t)g * (D / 32) * nkv + (int64_t)(D / 64) * 4 * owned_before(nrt_v, wave)) * kFragElems;
  st.n_pk = 2 * nks;
  st.n_pv = 16 * my_nrt;
  st.n_rv = (D / 64) * 4 * my_nrt;
  st.ntiles = ntiles;
  st.init(bm.off_rk + ((int64_t)g * nrt_k * NK + (int64_t)NK * owned_before(nrt_k, wave)) * kFragElems,
          NK * my_nrt_k);
  __bf16* ring = nullptr;
  int rs = 0, ws = 0;  // ring slots: next to read, next to fill
  if constexpr (NSLOT > 0) {
    ring = reinterpret_cast<__bf16*>(smem + a.ring_offset) + (size_t)wave * NSLOT * kFragElems;
#pragma unroll
    for (int k = 0; k < kDepth; ++k) lds_dma16(data_lane + st.next(), ring + k * kFragElems);
    ws = kDepth;
  }
  // the next fragment of the stream, in this lane's operand layout
  auto take = [&]() -> bf16x8 {
    if constexpr (NSLOT > 0) {
      wait_vmcnt<kDepth - 1>();
      const bf16x8 v = ld_bf16x8(ring + rs * kFragElems + lane * 8);
      lds_dma16(data_lane + st.next(), ring + ws * kFragElems);
      rs = rs + 1 == NSLOT ? 0 : rs + 1;
      ws = ws + 1 == NSLOT ? 0 : ws + 1;
      return v;
    } else {
      return ld_bf16x8(data_lane + st.next());
    }
  };

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
  __syncthreads();

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
    __syncthreads();
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
    __syncthreads();
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
  __syncthreads();  // every wave is done with qt / wl
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
    __syncthreads();
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
    __syncthreads();
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
  if constexpr (NSLOT > 0) wait_vmcnt<0>();  // no LDS write may land after the workgroup ends
}

template <int D, int MAX_RT, int NSLOT>
__global__ __launch_bounds__(kThreads, 1) void attend_kernel(AttendArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const WorkItem it = a.items[blockIdx.x];
  if (it.kind == kItemBlock) block_item<D, MAX_RT, NSLOT>(a, it, smem);
  else if (it.kind == kItemTail) tail_item<D>(a, it, smem);
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
  const size_t tail = (size_t)2 * kTailChunk * (head_dim + 8) * 2 +
                      ((size_t)kMaxGroup * head_dim + (size_t)kMaxGroup * kTailChunk) * 4 + kMaxGroup * 8;
  static_assert((size_t)kWaves * kMaxGroup * 128 * 4 <= (size_t)kTailChunk * (128 + 8) * 2,
                "tail value partials must fit over the staged K");
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
