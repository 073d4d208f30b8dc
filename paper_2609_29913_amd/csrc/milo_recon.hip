// Full-rank reconstruction of selected blocks (Sec. 4.5 inference path, Alg. 1
// full-rank reconstruction): K_b = P^K_b R^K_b and V_b = P^V_b R^V_b, one KV
// head's d columns and one 256-token tile per workgroup, written (keys as fp16,
// values as bf16) into the reconstruction buffer in the fragment layouts the
// attention kernel reads
// (P^K layout for K_{b,g}, P^V layout for V_{b,g}, both with rank d).
//
// A workgroup (8 waves) accumulates its 256 x d output tile over the block's
// rank in steps of 32 with v_mfma_f32_32x32x16_bf16, fp32 accumulation: every
// step stages the 256 x 32 slice of P and the 32 x d slice of R_g in LDS with
// the rank index contiguous (the MFMA contraction runs over the rank).  The
// cache stores P^K and R^V rank-contiguous already; P^V (token-contiguous, for
// the latent value pass) and R^K (dim-contiguous, for the query projection)
// are transposed on their way into LDS.  The next step's slices are loaded
// into registers while the current step's MFMAs run (two LDS buffers).  Every
// wave computes a 32-row-block x 32-column-block share of the tile: for V,
// tokens 64 (w % 4) .. +63 times dims (d / 2)(w / 4) .. +d/2; for K, the dim
// blocks b0 and b0 + d/64 (dims x and x + d/2, the pairs a rotary embedding
// turns together) of tokens 64 (w % 4) .. +63 with b0 = w / 4 at d = 128, of
// tokens 32 w .. +31 with b0 = 0 at d = 64.  For K it forms K^T = R^T P^T, so
// a lane's accumulators hold consecutive dims of one token and the tile goes
// to LDS as [token][dim] (pre-RoPE keys are rotated in fp32 on the way), for V
// it forms P R, giving consecutive tokens of one dim and an LDS tile
// [dim][token]; the packed fragments are then stored with one 16-byte store
// per lane.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "milo_internal.h"

namespace milo {
namespace {

typedef __bf16 bf16x8r __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4r __attribute__((ext_vector_type(4)));
typedef float f32x16r __attribute__((ext_vector_type(16)));
typedef _Float16 f16x4r __attribute__((ext_vector_type(4)));

constexpr int kReconThreads = 512;
constexpr int kStageStride = 40;  // bf16 row stride of a staged 32-rank slice (+8: conflict-free reads)

__device__ __forceinline__ f32x16r mfma32r(bf16x8r a, bf16x8r b, f32x16r c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// bytes of LDS the kernel uses for head dimension D
constexpr size_t recon_lds_bytes(int D) {
  const size_t stage = (size_t)2 * (kTile + D) * kStageStride * 2;
  const size_t out_k = (size_t)kTile * (D + 8) * 2, out_v = (size_t)D * (kTile + 8) * 2;
  const size_t out = out_k > out_v ? out_k : out_v;
  return stage > out ? stage : out;
}

// one task of side SIDE (0: K, 1: V)
template <int D, int SIDE>
__device__ __forceinline__ void recon_task(const ReconArgs& a, const ReconBlock& rb, int g, int t,
                                           unsigned char* smem) {
  constexpr int side = SIDE;
  // the wave's share: TI token blocks x TJ dim blocks of 32 (see above)
  constexpr int TI = (side == 0 && D == 64) ? 1 : 2;
  constexpr int TJ = side == 0 ? 2 : D / 64;
  const BlockMeta& bm = rb.src;
  const int nrt = (side ? bm.rv_pad : bm.rk_pad) >> 5;  // 32-rank steps
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 31, lhi = lane >> 5;
  const unsigned char* data = reinterpret_cast<const unsigned char*>(a.data);
  __bf16* sA = reinterpret_cast<__bf16*>(smem);      // [2][kTile][kStageStride]: P slice [token][rank]
  __bf16* sB = sA + 2 * kTile * kStageStride;         // [2][D][kStageStride]: R_g slice [dim][rank]

  // global -> registers for 32-rank step kc: two P chunks and (threads < 4 D) one
  // R chunk.  The fragment indices are split into per-task constants (set up
  // once) and a cheap per-step part: P^K and R^V advance by whole fragments per
  // step, P^V and R^K follow their rank-group / wave dealing (shifts only).
  const int f0 = tid >> 6, ln = tid & 63;  // chunk h covers fragment f0 + 8 h
  const unsigned char* pa_ptr[2];
  int pv_sig[2];
  const unsigned char* rb_ptr = data + 16 * ln;
  int pv0 = 0, T16 = 0, lgv = 0, rk0 = 0;
  if constexpr (side == 0) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int f = f0 + 8 * h;
      pa_ptr[h] = data + pk_frag(bm, kWaves * t + (f >> 1), f & 1) * (kFragElems * 2) + 16 * ln;
    }
    rk0 = (int)(bm.off_rk / kFragElems);
  } else {
    pv0 = (int)(bm.off_pv / kFragElems);
    T16 = bm.T_pad / 16;
    lgv = lg_rank_groups(nrt);
#pragma unroll
    for (int h = 0; h < 2; ++h) pv_sig[h] = 16 * t + f0 + 8 * h;
    if (tid < 4 * D) rb_ptr = data + rv_frag(bm, D, g, f0, 0) * (kFragElems * 2) + 16 * ln;
  }
  uint4 pa[2], rbv;
  auto load = [&](int kc) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (side == 0) {
        pa[h] = *reinterpret_cast<const uint4*>(pa_ptr[h] + (size_t)kc * 2 * (kFragElems * 2));
      } else {
        const int fr = pv_frag_split(pv0, T16, nrt, lgv, pv_sig[h], kc);
        pa[h] = *reinterpret_cast<const uint4*>(data + (int64_t)fr * (kFragElems * 2) + 16 * ln);
      }
    }
    if (tid < 4 * D) {
      if constexpr (side == 0) {
        const int fr = rk_frag_split(rk0, nrt, D / 16, g, kc, f0);
        rbv = *reinterpret_cast<const uint4*>(data + (int64_t)fr * (kFragElems * 2) + 16 * ln);
      } else {
        rbv = *reinterpret_cast<const uint4*>(rb_ptr + (size_t)kc * (kFragElems * 2));
      }
    }
  };
  // registers -> LDS buffer `buf` (rank contiguous)
  auto stage = [&](int buf) {
    __bf16* A = sA + buf * kTile * kStageStride;
    __bf16* B = sB + buf * D * kStageStride;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = tid + kReconThreads * h, f = q >> 6, ln = q & 63, m = ln & 31, c = ln >> 5;
      if (side == 0) {
        // P^K: lane (c, m) holds ranks 16 kap + 8 c .. +7 of token 32 tau + m
        *reinterpret_cast<uint4*>(A + (32 * (f >> 1) + m) * kStageStride + 16 * (f & 1) + 8 * c) = pa[h];
      } else {
        // P^V: lane (c, m) holds tokens 16 sig + 8 c .. +7 of rank 32 rho + m
        const __bf16* v = reinterpret_cast<const __bf16*>(&pa[h]);
#pragma unroll
        for (int e = 0; e < 8; ++e) A[(16 * f + 8 * c + e) * kStageStride + m] = v[e];
      }
    }
    if (tid < 4 * D) {
      const int f = tid >> 6, ln = tid & 63;
      if (side == 0) {
        // R^K: lane (c, m) holds dims 16 kap + 8 c .. +7 (of head g) at rank 32 rho + m
        const int m = ln & 31, c = ln >> 5;
        const __bf16* v = reinterpret_cast<const __bf16*>(&rbv);
#pragma unroll
        for (int e = 0; e < 8; ++e) B[(16 * f + 8 * c + e) * kStageStride + m] = v[e];
      } else {
        // R^V: lane 16 qq + n holds ranks 32 kap + 8 qq .. +7 at dim 16 ds + n
        const int n = ln & 15, qq = ln >> 4;
        *reinterpret_cast<uint4*>(B + (16 * f + n) * kStageStride + 8 * qq) = rbv;
      }
    }
  };

  auto tok_block = [&](int i) { return TI == 2 ? 2 * (wave & 3) + i : wave; };
  auto dim_block = [&](int j) {
    return side == 0 ? (D == 128 ? (wave >> 2) : 0) + (D / 64) * j : (D / 64) * (wave >> 2) + j;
  };
  f32x16r acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f32x16r{};
  load(0);
  stage(0);
  __syncthreads();
  for (int kc = 0; kc < nrt; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nrt) load(kc + 1);
    const __bf16* A = sA + buf * kTile * kStageStride;
    const __bf16* B = sB + buf * D * kStageStride;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8r af[TI], bfr[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i)
        af[i] = *reinterpret_cast<const bf16x8r*>(A + (32 * tok_block(i) + lrow) * kStageStride + 16 * kk + 8 * lhi);
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8r*>(B + (32 * dim_block(j) + lrow) * kStageStride + 16 * kk + 8 * lhi);
      if (side == 0) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) acc[i][j] = mfma32r(bfr[j], af[i], acc[i][j]);  // K^T: [dim][token]
      } else {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) acc[i][j] = mfma32r(af[i], bfr[j], acc[i][j]);  // V: [token][dim]
      }
    }
    if (kc + 1 < nrt) stage(buf ^ 1);  // the other buffer: its last readers passed the previous barrier
    __syncthreads();
  }

  // pre-RoPE keys: lane (lhi, lrow) holds dims x = 32 b0 + 8 jj + 4 lhi + u and
  // x + d/2 of token 32 tok_block(i) + lrow of tile t, at position
  // p = pos0 + 256 t + that token; the pair turns by the angle p w_x, formed in
  // turns in fp64 (exact to ~1e-9 turns for int32 positions), reduced to [0, 1)
  // and evaluated by the hardware's sine and cosine of an angle in turns (fp32;
  // error below 1.3e-7 over [0, 1), measured on gfx950)
  if constexpr (side == 0) {
    if (rb.pos0 >= 0) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int x = 32 * dim_block(0) + 8 * jj + 4 * lhi;  // < d / 2
        const double2 w01 = *reinterpret_cast<const double2*>(a.rope_turns + x);
        const double2 w23 = *reinterpret_cast<const double2*>(a.rope_turns + x + 2);
        const double w[4] = {w01.x, w01.y, w23.x, w23.y};
#pragma unroll
        for (int i = 0; i < TI; ++i) {
          const double p = (double)(rb.pos0 + kTile * t + 32 * tok_block(i) + lrow);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const double turns = p * w[u];
            const float r = (float)(turns - floor(turns));
            const float sn = __builtin_amdgcn_sinf(r), c = __builtin_amdgcn_cosf(r);
            const float k0 = acc[i][0][4 * jj + u], k1 = acc[i][1][4 * jj + u];
            acc[i][0][4 * jj + u] = k0 * c - k1 * sn;
            acc[i][1][4 * jj + u] = k1 * c + k0 * sn;
          }
        }
      }
    }
  }

  // the tile as bf16 in LDS (all staging reads are done: the loop ended on a barrier)
  __bf16* O = reinterpret_cast<__bf16*>(smem);
  constexpr int kOK = D + 8, kOV = kTile + 8;  // row strides: K [token][dim], V [dim][token]
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int tok_blk = 32 * tok_block(i), dim_blk = 32 * dim_block(j);
        if (side == 0) {
          // keys as fp16 (saturated at +-65504): 8x finer than bf16 where the
          // score of a peaked softmax needs it; rows: dims 8 jj + 4 lhi + u of
          // the block, column: token lrow
          f16x4r v;
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = (_Float16)fminf(fmaxf(acc[i][j][4 * jj + u], -65504.f), 65504.f);
          *reinterpret_cast<f16x4r*>(O + (tok_blk + lrow) * kOK + dim_blk + 8 * jj + 4 * lhi) = v;
        } else {  // values as bf16; rows: tokens 8 jj + 4 lhi + u, column: dim lrow
          bf16x4r v;
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = (__bf16)acc[i][j][4 * jj + u];
          *reinterpret_cast<bf16x4r*>(O + (dim_blk + lrow) * kOV + tok_blk + 8 * jj + 4 * lhi) = v;
        }
      }
  __syncthreads();

  // packed stores: 32 D chunks of 16 bytes (D / 2 fragments of 64 lanes).  With
  // rank d every rank group of the P^V layout owns one rank tile (v_segments:
  // 2 token segments for d = 128, 4 for d = 64), so fragment (sig, rho) sits at
  // rho T_pad / 16 + sig.
  static_assert(kWaves / v_segments(D / 32) == D / 32, "one rank tile per rank group at rank d");
  const BlockMeta dm = dense_meta(bm, rb.dst, g, D);
  const int tiles_all = bm.T_pad / kTile;
  unsigned char* out = reinterpret_cast<unsigned char*>(a.recon);
  for (int q = tid; q < 32 * D; q += kReconThreads) {
    const int f = q >> 6, ln = q & 63, m = ln & 31, c = ln >> 5;
    int64_t frag;
    uint4 v;
    if constexpr (side == 0) {
      // K_{b,g} in the P^K layout: fragment (tau = 8 t + w, kap), lane (c, m) = dims 16 kap + 8 c .. +7 of token 32 w + m
      const int w = f / (D / 16), kap = f % (D / 16);
      frag = dm.off_pk / kFragElems + ((int64_t)w * tiles_all + t) * (D / 16) + kap;
      v = *reinterpret_cast<const uint4*>(O + (32 * w + m) * kOK + 16 * kap + 8 * c);
    } else {
      // V_{b,g} in the P^V layout: fragment (sig = 16 t + s, rho), lane (c, m) = tokens 16 s + 8 c .. +7 of dim 32 rho + m
      const int s = f / (D / 32), rho = f % (D / 32);
      frag = dm.off_pv / kFragElems + (int64_t)rho * (bm.T_pad / 16) + 16 * t + s;
      v = *reinterpret_cast<const uint4*>(O + (32 * rho + m) * kOV + 16 * s + 8 * c);
    }
    *reinterpret_cast<uint4*>(out + frag * (kFragElems * 2) + 16 * ln) = v;
  }
}

template <int D>
__global__ __launch_bounds__(kReconThreads) void recon_kernel(ReconArgs a) {
  static_assert(D == 64 || D == 128, "head dimension");
  extern __shared__ __align__(16) unsigned char smem[];
  const int2 task = a.tasks[blockIdx.x];
  if (task.x < 0) return;
  const ReconBlock rb = a.blocks[task.x];
  const int g = (task.y >> 1) & 127, t = task.y >> 8;
  if (task.y & 1) recon_task<D, 1>(a, rb, g, t, smem);
  else recon_task<D, 0>(a, rb, g, t, smem);
}

// One wave per packed fragment of a prefill chunk's shared tail (K of every
// head in the P^K layout of rank d, V in the P^V layout, as the reconstruction
// kernel stores them); lane (c, m) gathers its 8 elements.
template <int D>
__global__ __launch_bounds__(256) void pack_tail_kernel(TailPackArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t per_side = (int64_t)a.T_pad * D / kFragElems;
  const int64_t f = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (f >= 2 * a.n_kv * per_side) return;
  const int g = (int)(f / (2 * per_side)), side = (int)((f / per_side) & 1);
  const int64_t fr = f % per_side;
  const int m = lane & 31, c = lane >> 5;
  const int64_t rs = (int64_t)a.n_kv * D;  // tail row stride
  uint4 v;
  __bf16* ve = reinterpret_cast<__bf16*>(&v);
  if (side == 0) {
    // fragment (tau = 8 t + w, kap) of the P^K layout: dims 16 kap + 8 c .. +7 of token 32 tau + m
    constexpr int nks = D / 16;
    const int tiles = a.T_pad / kTile;
    const int kap = (int)(fr % nks), t = (int)((fr / nks) % tiles), w = (int)(fr / ((int64_t)nks * tiles));
    const int row = 32 * (kWaves * t + w) + m;
    if (row < a.rows) {
      // keys as fp16, as the reconstruction kernel stores them (saturated at +-65504)
      const uint4 kb = *reinterpret_cast<const uint4*>(a.tail_k + row * rs + (int64_t)g * D + 16 * kap + 8 * c);
      const __bf16* kv = reinterpret_cast<const __bf16*>(&kb);
      _Float16* hv = reinterpret_cast<_Float16*>(&v);
#pragma unroll
      for (int e = 0; e < 8; ++e) hv[e] = (_Float16)fminf(fmaxf((float)kv[e], -65504.f), 65504.f);
    } else {
      v = make_uint4(0, 0, 0, 0);
    }
  } else {
    // fragment rho T_pad / 16 + sig of the P^V layout at rank d: tokens 16 sig + 8 c .. +7 of dim 32 rho + m
    const int T16 = a.T_pad / 16;
    const int rho = (int)(fr / T16), sig = (int)(fr % T16);
    const uint16_t* src = a.tail_v + (int64_t)g * D + 32 * rho + m;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = 16 * sig + 8 * c + e;
      const uint16_t u = row < a.rows ? src[row * rs] : (uint16_t)0;
      ve[e] = *reinterpret_cast<const __bf16*>(&u);
    }
  }
  uint16_t* dst = a.recon + a.region + ((int64_t)g * 2 + side) * a.T_pad * D + fr * kFragElems;
  *reinterpret_cast<uint4*>(dst + 8 * lane) = v;
}

template <int D>
hipError_t launch_recon_t(const ReconArgs& a, int n_tasks, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const size_t lds = recon_lds_bytes(D);
  static bool attr_set = false;
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&recon_kernel<D>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipExtLaunchKernelGGL(recon_kernel<D>, dim3(n_tasks), dim3(kReconThreads), (uint32_t)lds, s, e0, e1, 0, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pack_tail(const TailPackArgs& a, int head_dim, hipStream_t s) {
  const int64_t frags = 2LL * a.n_kv * a.T_pad * head_dim / kFragElems;
  const dim3 grid((unsigned)((frags + 3) / 4));
  if (head_dim == 64) hipLaunchKernelGGL(pack_tail_kernel<64>, grid, dim3(256), 0, s, a);
  else if (head_dim == 128) hipLaunchKernelGGL(pack_tail_kernel<128>, grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_recon(const ReconArgs& a, int head_dim, int n_tasks, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (n_tasks <= 0) return hipSuccess;
  if (head_dim == 64) return launch_recon_t<64>(a, n_tasks, s, e0, e1);
  if (head_dim == 128) return launch_recon_t<128>(a, n_tasks, s, e0, e1);
  return hipErrorInvalidValue;
}

}  // namespace milo
