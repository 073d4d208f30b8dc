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
//     tail item (request i, KV head g, chunk of the request's own KV):
//       plain attention of the group's query heads over the chunk (VALU)
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

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

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
// tokens [t0, t0 + nt) of that request's uncompressed KV.
// ---------------------------------------------------------------------------
template <int D>
__device__ void tail_item(const AttendArgs& a, int4 task, unsigned char* smem) {
  constexpr int kParts = kThreads / D;
  const int i = -1 - task.x, slot = task.y, g = task.z, chunk = task.w;
  const int G = a.G, TC = a.tail_chunk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int t0 = chunk * TC;
  const int nt = min(TC, a.tail_len[i] - t0);
  float* qs = reinterpret_cast<float*>(smem);   // [G][D]
  float* sc = qs + G * D;                       // [G][TC]
  float2* ml = reinterpret_cast<float2*>(sc + G * TC);  // [G]
  float* op = reinterpret_cast<float*>(ml + kMaxGroup);  // [kParts][G][D]

  for (int x = tid; x < G * D; x += kThreads) {
    const int hh = x / D, j = x % D;
    qs[x] = bf16_to_f32(a.q[((int64_t)i * a.H_q + g * G + hh) * D + j]) * a.qscale;
  }
  __syncthreads();
  const int64_t rstride = (int64_t)a.H_kv * D;
  const uint16_t* kb = a.tail_k + ((int64_t)i * a.tail_cap + t0) * rstride + (int64_t)g * D;
  const uint16_t* vb = a.tail_v + ((int64_t)i * a.tail_cap + t0) * rstride + (int64_t)g * D;
  for (int x = tid; x < nt * G; x += kThreads) {
    const int t = x / G, hh = x % G;
    const uint16_t* kr = kb + t * rstride;
    const float* qh = qs + hh * D;
    float acc = 0.f;
#pragma unroll 8
    for (int j = 0; j < D; j += 8) {
      const uint4 raw = *reinterpret_cast<const uint4*>(kr + j);
      const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        acc += __uint_as_float(w[u] << 16) * qh[j + 2 * u];
        acc += __uint_as_float(w[u] & 0xffff0000u) * qh[j + 2 * u + 1];
      }
    }
    sc[hh * TC + t] = acc;
  }
  __syncthreads();
  for (int hh = wave; hh < G; hh += kWaves) {
    float mx = -INFINITY;
    for (int t = lane; t < nt; t += 64) mx = fmaxf(mx, sc[hh * TC + t]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.f;
    for (int t = lane; t < nt; t += 64) {
      const float w = fast_exp2(sc[hh * TC + t] - mx);
      sc[hh * TC + t] = w;
      sum += w;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) ml[hh] = make_float2(mx, sum);
  }
  __syncthreads();
  const int j = tid % D, part = tid / D;
  float acc[kMaxGroup];
#pragma unroll
  for (int hh = 0; hh < kMaxGroup; ++hh) acc[hh] = 0.f;
  for (int t = part; t < nt; t += kParts) {
    const float v = bf16_to_f32(vb[t * rstride + j]);
#pragma unroll
    for (int hh = 0; hh < kMaxGroup; ++hh)
      if (hh < G) acc[hh] += sc[hh * TC + t] * v;
  }
#pragma unroll
  for (int hh = 0; hh < kMaxGroup; ++hh)
    if (hh < G) op[(part * G + hh) * D + j] = acc[hh];
  __syncthreads();
  for (int x = tid; x < G * D; x += kThreads) {
    const int hh = x / D, jj = x % D;
    float s = 0.f;
#pragma unroll
    for (int p = 0; p < kParts; ++p) s += op[(p * G + hh) * D + jj];
    const int64_t col = (int64_t)i * a.H_q + g * G + hh;
    a.part_o[(col * a.n_slots + slot) * D + jj] = s;
    if (jj == 0) a.part_ml[col * a.n_slots + slot] = ml[hh];
  }
}

// ---------------------------------------------------------------------------
// Block work item: latent-space attention of one 64-column tile of the query
// columns of KV head g over all tokens of block b.
// ---------------------------------------------------------------------------
template <int D, int MAX_RT>
__device__ void block_item(const AttendArgs& a, int4 task, unsigned char* smem) {
  const BlockMeta bm = a.meta[task.x];
  const int slot = task.y, g = task.z, c0 = task.w * kCols;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  const int G = a.G, ncg = a.n_q * G;
  const int qsd = a.qt_stride;
  const int nrt_k = bm.rk_pad >> 5, nks = bm.rk_pad >> 4;
  const int nrt_v = bm.rv_pad >> 5;
  __bf16* qt = reinterpret_cast<__bf16*>(smem);              // [kCols][qsd]
  __bf16* wl = qt + kCols * qsd;                               // [kCols][kWStride]
  float* red = reinterpret_cast<float*>(wl + kCols * kWStride);  // [kWaves][kCols]

  // ---- projection: Qt[rank][col] (stored [col][rank]) ----
  {
    constexpr int NK = D / 16;
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
    const uint16_t* rkb = a.data + bm.off_rk + (int64_t)g * nrt_k * NK * kFragElems + lane * 8;
    for (int rt = wave; rt < nrt_k; rt += kWaves) {
      f32x16 acc0 = {}, acc1 = {};
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        const bf16x8 af = ld_bf16x8(rkb + (int64_t)(rt * NK + k) * kFragElems);
        acc0 = mfma32(af, qf[k][0], acc0);
        acc1 = mfma32(af, qf[k][1], acc1);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 v0, v1;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          v0[u] = (__bf16)(acc0[4 * j + u] * a.qscale);
          v1[u] = (__bf16)(acc1[4 * j + u] * a.qscale);
        }
        const int r = 32 * rt + 8 * j + 4 * lhi;
        *reinterpret_cast<bf16x4*>(qt + lrow * qsd + r) = v0;
        *reinterpret_cast<bf16x4*>(qt + (32 + lrow) * qsd + r) = v1;
      }
    }
  }
  __syncthreads();

  // ---- scores, online softmax, latent V ----
  const int T = bm.T, T32 = bm.T_pad >> 5, T16 = bm.T_pad >> 4;
  const uint16_t* pkb = a.data + bm.off_pk + lane * 8;
  const uint16_t* pvb = a.data + bm.off_pv + lane * 8;
  f32x16 oacc[MAX_RT][2];
#pragma unroll
  for (int r = 0; r < MAX_RT; ++r) oacc[r][0] = oacc[r][1] = f32x16{};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};

  for (int t0 = 0; t0 < T; t0 += kTile) {
    const int tw = t0 + wave * kTokWave;
    const int tau0 = tw >> 5;
    f32x16 s[2][2];
    s[0][0] = s[0][1] = s[1][0] = s[1][1] = f32x16{};
    const bool v0 = tau0 < T32, v1 = tau0 + 1 < T32;
    const uint16_t* pk0 = pkb + (int64_t)tau0 * nks * kFragElems;
    const uint16_t* pk1 = pk0 + (int64_t)nks * kFragElems;
    const __bf16* qr0 = qt + lrow * qsd + 8 * lhi;
    const __bf16* qr1 = qt + (32 + lrow) * qsd + 8 * lhi;
    if (v0) {
#pragma unroll 4
      for (int k = 0; k < nks; ++k) {
        const bf16x8 b0 = *reinterpret_cast<const bf16x8*>(qr0 + 16 * k);
        const bf16x8 b1 = *reinterpret_cast<const bf16x8*>(qr1 + 16 * k);
        const bf16x8 a0 = ld_bf16x8(pk0 + (int64_t)k * kFragElems);
        s[0][0] = mfma32(a0, b0, s[0][0]);
        s[0][1] = mfma32(a0, b1, s[0][1]);
        if (v1) {
          const bf16x8 a1 = ld_bf16x8(pk1 + (int64_t)k * kFragElems);
          s[1][0] = mfma32(a1, b0, s[1][0]);
          s[1][1] = mfma32(a1, b1, s[1][1]);
        }
      }
    }
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
    const int sg0 = t0 >> 4;
    const int nsg = min(kTile / 16, T16 - sg0);
    const __bf16* wr0 = wl + lrow * kWStride + 8 * lhi;
    const __bf16* wr1 = wl + (32 + lrow) * kWStride + 8 * lhi;
    for (int sg = 0; sg < nsg; ++sg) {
      const bf16x8 w0 = *reinterpret_cast<const bf16x8*>(wr0 + 16 * sg);
      const bf16x8 w1 = *reinterpret_cast<const bf16x8*>(wr1 + 16 * sg);
      const uint16_t* pvs = pvb + (int64_t)(sg0 + sg) * nrt_v * kFragElems;
#pragma unroll
      for (int r = 0; r < MAX_RT; ++r) {
        const int rt = wave + kWaves * r;
        if (rt < nrt_v) {
          const bf16x8 af = ld_bf16x8(pvs + (int64_t)rt * kFragElems);
          oacc[r][0] = mfma32(af, w0, oacc[r][0]);
          oacc[r][1] = mfma32(af, w1, oacc[r][1]);
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
  const int nkv = bm.rv_pad >> 4;
  const uint16_t* rvb = a.data + bm.off_rv + (int64_t)g * (D / 32) * nkv * kFragElems + lane * 8;
#pragma unroll
  for (int pass = 0; pass < D / 64; ++pass) {
    f32x16 acc[2][2];
    acc[0][0] = acc[0][1] = acc[1][0] = acc[1][1] = f32x16{};
#pragma unroll
    for (int r = 0; r < MAX_RT; ++r) {
      const int rt = wave + kWaves * r;
      if (rt < nrt_v) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          bf16x8 b0, b1;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            b0[e] = (__bf16)oacc[r][0][8 * half + e];
            b1[e] = (__bf16)oacc[r][1][8 * half + e];
          }
          const int kv = 2 * rt + half;
#pragma unroll
          for (int dt = 0; dt < 2; ++dt) {
            const int dl = 2 * pass + dt;
            const bf16x8 af = ld_bf16x8(rvb + (int64_t)(dl * nkv + kv) * kFragElems);
            acc[dt][0] = mfma32(af, b0, acc[dt][0]);
            acc[dt][1] = mfma32(af, b1, acc[dt][1]);
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
}

template <int D, int MAX_RT>
__global__ __launch_bounds__(kThreads, 1) void attend_kernel(AttendArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int4 task = a.tasks[blockIdx.x];
  if (task.x == kEmptyTask) return;
  if (task.x < 0) {
    tail_item<D>(a, task, smem);
    return;
  }
  block_item<D, MAX_RT>(a, task, smem);
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge: one workgroup (D threads) per query column (i, h).
// Slots [0, n_sel) are the selected blocks, then request i's tail chunks.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(D) void merge_kernel(MergeArgs a) {
  __shared__ float red[D / 64];
  const int col = blockIdx.x, j = threadIdx.x;
  const int i = col / a.H_q;
  const int n_valid = a.n_sel + (a.tail_len[i] + a.tail_chunk - 1) / a.tail_chunk;
  const float2* ml = a.part_ml + (int64_t)col * a.n_slots;
  float mx = -INFINITY;
  for (int s = j; s < n_valid; s += D) mx = fmaxf(mx, ml[s].x);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((j & 63) == 0) red[j >> 6] = mx;
  __syncthreads();
  mx = red[0];
#pragma unroll
  for (int w = 1; w < D / 64; ++w) mx = fmaxf(mx, red[w]);
  float num = 0.f, den = 0.f;
  const float* po = a.part_o + (int64_t)col * a.n_slots * D + j;
  for (int s = 0; s < n_valid; ++s) {
    const float2 v = ml[s];
    const float f = fast_exp2(v.x - mx);
    den += v.y * f;
    num += po[(int64_t)s * D] * f;
  }
  a.out[(int64_t)col * D + j] = num / den;
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

size_t attend_lds_bytes(int head_dim, int rk_pad_max, int G, int tail_chunk) {
  const size_t qsd = (size_t)rk_pad_max + 8;
  const size_t loop = kCols * qsd * 2 + (size_t)kCols * kWStride * 2 + (size_t)kWaves * kCols * 4;
  const size_t epi = ((size_t)kWaves * kCols * kORow + (size_t)kWaves * kCols) * 4;
  const size_t tail = ((size_t)G * head_dim + (size_t)G * tail_chunk) * 4 + kMaxGroup * 8 +
                      (size_t)(kThreads / head_dim) * G * head_dim * 4;
  size_t m = loop > epi ? loop : epi;
  return m > tail ? m : tail;
}

template <int D, int MAX_RT>
static hipError_t launch_attend_t(const AttendArgs& a, int grid, size_t lds, hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_kernel<D, MAX_RT>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((attend_kernel<D, MAX_RT>), dim3(grid), dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_attend_d(const AttendArgs& a, int max_rt, int grid, size_t lds, hipStream_t s) {
  switch (max_rt) {
    case 1: return launch_attend_t<D, 1>(a, grid, lds, s);
    case 2: return launch_attend_t<D, 2>(a, grid, lds, s);
    case 4: return launch_attend_t<D, 4>(a, grid, lds, s);
    case 6: return launch_attend_t<D, 6>(a, grid, lds, s);
    case 8: return launch_attend_t<D, 8>(a, grid, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attend(const AttendArgs& a, int head_dim, int max_rt, int grid, size_t lds_bytes,
                         hipStream_t s) {
  if (grid == 0) return hipSuccess;
  if (head_dim == 64) return launch_attend_d<64>(a, max_rt, grid, lds_bytes, s);
  if (head_dim == 128) return launch_attend_d<128>(a, max_rt, grid, lds_bytes, s);
  return hipErrorInvalidValue;
}

hipError_t launch_merge(const MergeArgs& a, int head_dim, int n_cols, hipStream_t s) {
  if (head_dim == 64) {
    hipLaunchKernelGGL(merge_kernel<64>, dim3(n_cols), dim3(64), 0, s, a);
  } else if (head_dim == 128) {
    hipLaunchKernelGGL(merge_kernel<128>, dim3(n_cols), dim3(128), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace milo
