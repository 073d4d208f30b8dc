// Host side of the C ABI in include/milo.h: argument validation, the packed
// cache (Sec. 4.2 factors stored per block with per-block ranks, Sec. 4.3),
// the per-call work plan and the kernel launches of one decode step
// (Alg. 1 inference stage: attention over the selected blocks plus the
// request's own KV).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <vector>

#include "milo.h"
#include "milo_attend.h"
#include "milo_internal.h"
#include "milo_plan.h"

using namespace milo;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
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

constexpr int64_t kAlignElems = kFragElems;  // every packed factor starts on a whole fragment
constexpr int64_t kPackStageElems = int64_t(64) << 20;  // staging of host factors (128 MiB of bf16)

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

int64_t env_byte_cap() {
  const char* s = std::getenv("MILO_MAX_DEVICE_BYTES");
  if (!s || !*s) return -1;
  return std::strtoll(s, nullptr, 10);
}

// LDS bytes a workgroup program may use at most, from MILO_MAX_PROGRAM_BYTES
// (unset: no cap beyond what LDS leaves).  A small cap splits a step's work
// over several attention launches; it exists so that path can be exercised.
int64_t env_program_cap() {
  const char* s = std::getenv("MILO_MAX_PROGRAM_BYTES");
  if (!s || !*s) return -1;
  return std::strtoll(s, nullptr, 10);
}

// Timing hooks (measurement only).
struct TimingState {
  std::mutex mu;
  bool enabled = false;
  std::vector<hipEvent_t> pool;
  std::vector<hipEvent_t> recorded;  // groups of 4: attend kernel start / end, merge kernel start / end
  std::vector<hipEvent_t> recon_recorded;  // pairs: reconstruction kernel start / end
};
TimingState g_timing;

}  // namespace

struct milo_cache {
  int device = -1;
  uint64_t serial = 0;  // distinct for every cache of the process (plan keys)
  bool p_int8 = false;  // P^K / P^V stored as INT8 codes with per-token scales
  int n_blocks = 0, n_kv = 0, d = 0;
  std::vector<int32_t> T, rk, rv;
  std::vector<BlockMeta> meta;
  uint16_t* data = nullptr;
  int64_t data_elems = 0;
  // per-call workspace of milo_attend_decode / milo_attend_prefill
  float* part_o = nullptr;
  float2* part_ml = nullptr;
  int64_t part_cols_slots = 0;  // capacity in (column, slot) pairs
  unsigned char* plan_d = nullptr;       // program table + programs of the attention launches
  unsigned char* plan_pinned = nullptr;  // staging copy for the upload
  int64_t plan_cap = 0;
  hipEvent_t plan_evt = nullptr;         // recorded after the last upload from plan_pinned
  bool plan_evt_live = false;
  int32_t* tail_len_d = nullptr;         // tail lengths of batches above kInlineTails requests
  int64_t tail_len_cap = 0;
  int32_t path = MILO_PATH_LATENT;       // milo_cache_set_path
  unsigned char* recon_raw = nullptr;    // reconstruction buffer (allocation)
  uint16_t* recon_d = nullptr;           // its start, a whole number of fragments from `data`
  int64_t recon_cap = 0;                 // capacity in bf16 elements
  PlanState plan;                        // the plan of the previous call
  // pre-RoPE keys (milo_cache_set_rope): first-token position per block, and
  // the rotation table the reconstruction kernel reads
  std::vector<int32_t> rope_pos;         // empty: keys are attended as stored
  double* rope_d = nullptr;              // [d/2] w_j / (2 pi)
  int32_t rope_gen = 0;                  // changes with every setting (plan keys)
};

namespace {

FactorGeom geom_of(const milo_cache& c, int b, int which) {
  FactorGeom f{};
  f.kind = which;
  f.n_kv = c.n_kv;
  f.d = c.d;
  const int D = c.n_kv * c.d;
  f.T_pad = (int)round_up(c.T[b], kTile);
  switch (which) {
    case kPK: f.rows = c.T[b]; f.cols = c.rk[b]; f.r_pad = (int)round_up(c.rk[b], 32); break;
    case kRK: f.rows = c.rk[b]; f.cols = D; f.r_pad = (int)round_up(c.rk[b], 32); break;
    case kPV: f.rows = c.T[b]; f.cols = c.rv[b]; f.r_pad = (int)round_up(c.rv[b], 32); break;
    default:  f.rows = c.rv[b]; f.cols = D; f.r_pad = (int)round_up(c.rv[b], 32); break;
  }
  return f;
}

int64_t factor_offset(const BlockMeta& m, int which) {
  switch (which) {
    case kPK: return m.off_pk;
    case kRK: return m.off_rk;
    case kPV: return m.off_pv;
    default:  return m.off_rv;
  }
}

void destroy(milo_cache* c) {
  if (!c) return;
  if (c->device >= 0) {
    int cur = -1;
    if (hipGetDevice(&cur) == hipSuccess && cur != c->device) (void)hipSetDevice(c->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(c->data);
    (void)hipFree(c->part_o);
    (void)hipFree(c->part_ml);
    (void)hipFree(c->plan_d);
    (void)hipFree(c->tail_len_d);
    (void)hipFree(c->recon_raw);
    (void)hipFree(c->rope_d);
    (void)hipHostFree(c->plan_pinned);
    if (c->plan_evt) (void)hipEventDestroy(c->plan_evt);
    if (cur >= 0 && cur != c->device) (void)hipSetDevice(cur);
  }
  delete c;
}

}  // namespace

namespace milo {
void clear_error() { g_err.clear(); }
int report_error(int code, const char* msg) { return fail(code, "%s", msg); }
bool timing_enabled() {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  return g_timing.enabled;
}
}  // namespace milo

extern "C" {

const char* milo_last_error(void) { return g_err.c_str(); }

int milo_cache_create(const milo_cache_desc* desc, const uint16_t* const* pk, const uint16_t* const* rk,
                      const uint16_t* const* pv, const uint16_t* const* rv, int src_on_device,
                      void* hip_stream, milo_cache** out) {
  g_err.clear();
  if (!out) return fail(MILO_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!desc) return fail(MILO_ERR_INVALID_ARG, "desc is NULL");
  if (desc->n_blocks < 1) return fail(MILO_ERR_INVALID_ARG, "n_blocks must be >= 1 (got %d)", desc->n_blocks);
  if (desc->n_kv_heads < 1) return fail(MILO_ERR_INVALID_ARG, "n_kv_heads must be >= 1");
  if (desc->head_dim != 64 && desc->head_dim != 128)
    return fail(MILO_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", desc->head_dim);
  if (!desc->block_tokens || !desc->rank_k || !desc->rank_v)
    return fail(MILO_ERR_INVALID_ARG, "block_tokens / rank_k / rank_v must be non-NULL");
  if (!pk || !rk || !pv || !rv) return fail(MILO_ERR_INVALID_ARG, "factor pointer arrays must be non-NULL");
  if (src_on_device != 0 && src_on_device != 1) return fail(MILO_ERR_INVALID_ARG, "src_on_device must be 0 or 1");
  if (desc->p_format != MILO_P_BF16 && desc->p_format != MILO_P_INT8)
    return fail(MILO_ERR_INVALID_ARG, "p_format must be MILO_P_BF16 or MILO_P_INT8 (got %d)", desc->p_format);
  const bool i8 = desc->p_format == MILO_P_INT8;
  const int64_t D = (int64_t)desc->n_kv_heads * desc->head_dim;
  for (int b = 0; b < desc->n_blocks; ++b) {
    const int T = desc->block_tokens[b], a = desc->rank_k[b], v = desc->rank_v[b];
    if (T < 1) return fail(MILO_ERR_INVALID_ARG, "block %d: T_b must be >= 1 (got %d)", b, T);
    if (a < 1 || a > T || a > D || v < 1 || v > T || v > D)
      return fail(MILO_ERR_INVALID_ARG, "block %d: ranks (%d, %d) must lie in [1, min(T_b=%d, H_kv*d=%lld)]",
                  b, a, v, T, (long long)D);
    const int rmax = i8 ? kMaxRank : kMaxStoredRank;  // INT8 blocks attend latent only
    if (a > rmax || v > rmax)
      return fail(MILO_ERR_UNSUPPORTED, "block %d: rank above the supported maximum %d", b, rmax);
    if (!pk[b] || !rk[b] || !pv[b] || !rv[b]) return fail(MILO_ERR_INVALID_ARG, "block %d: NULL factor", b);
  }

  static std::atomic<uint64_t> next_serial{1};
  milo_cache* c = new milo_cache();
  c->serial = next_serial.fetch_add(1);
  c->n_blocks = desc->n_blocks;
  c->p_int8 = i8;
  c->n_kv = desc->n_kv_heads;
  c->d = desc->head_dim;
  c->T.assign(desc->block_tokens, desc->block_tokens + c->n_blocks);
  c->rk.assign(desc->rank_k, desc->rank_k + c->n_blocks);
  c->rv.assign(desc->rank_v, desc->rank_v + c->n_blocks);
  c->meta.resize(c->n_blocks);
  int64_t off = 0, max_src = 0, max_tpad = 0, total_src = 0;
  for (int b = 0; b < c->n_blocks; ++b) {
    BlockMeta& m = c->meta[b];
    m.T = c->T[b];
    m.T_pad = (int)round_up(c->T[b], kTile);
    m.rk_pad = (int)round_up(c->rk[b], 32);
    m.rv_pad = (int)round_up(c->rv[b], 32);
    int64_t* offs[4] = {&m.off_pk, &m.off_rk, &m.off_pv, &m.off_rv};
    for (int w = 0; w < 4; ++w) {
      const FactorGeom f = geom_of(*c, b, w);
      *offs[w] = off;
      // INT8 P factors: one byte per code, and after P^V the block's scale units
      int64_t elems = frag_count(f) * kFragElems;
      if (i8 && w == kPK) elems = i8_factor_bytes(m.T_pad, m.rk_pad) / 2;
      if (i8 && w == kPV) elems = i8_factor_bytes(m.T_pad, m.rv_pad) / 2 + i8_scale_bytes(m.T_pad) / 2;
      off = round_up(off + elems, kAlignElems);
      max_src = std::max<int64_t>(max_src, (int64_t)f.rows * f.cols);
      total_src += round_up((int64_t)f.rows * f.cols, 8);
    }
    max_tpad = std::max<int64_t>(max_tpad, m.T_pad);
  }
  c->data_elems = off;
  if (off / kFragElems >= ((int64_t)1 << 31)) {
    delete c;
    return fail(MILO_ERR_UNSUPPORTED, "cache of %lld elements exceeds the 2^31-fragment index range", (long long)off);
  }
  // host sources go through a staging buffer: one factor at a time for INT8
  // (whose scales need a kernel per factor), else as many as kPackStageElems hold
  const int64_t stage_elems =
      src_on_device ? 0
      : i8          ? max_src
                    : std::max<int64_t>(round_up(max_src, 8), std::min<int64_t>(total_src, kPackStageElems));
  const int64_t need = off * 2 + stage_elems * 2;
  const int64_t cap = env_byte_cap();
  if (cap >= 0 && need > cap) {
    delete c;
    return fail(MILO_ERR_OUT_OF_MEMORY, "cache needs %lld device bytes, above MILO_MAX_DEVICE_BYTES=%lld",
                (long long)need, (long long)cap);
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  uint16_t* staging = nullptr;
  float* i8_tmp = nullptr;  // INT8: K and V row scales of the block being packed, then a flag
  auto cleanup_fail = [&](int code) {
    if (staging) (void)hipFree(staging);
    if (i8_tmp) (void)hipFree(i8_tmp);
    destroy(c);
    return code;
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) { c->device = -1; return cleanup_fail(hip_fail(e, "hipGetDevice")); }
  if ((e = hipMalloc(&c->data, (size_t)c->data_elems * 2)) != hipSuccess)
    return cleanup_fail(hip_fail(e, "hipMalloc(packed factors)"));
  if (!src_on_device && (e = hipMalloc(&staging, (size_t)stage_elems * 2)) != hipSuccess)
    return cleanup_fail(hip_fail(e, "hipMalloc(staging)"));
  float *ks = nullptr, *vs = nullptr;
  int* bad = nullptr;
  if (i8) {
    if ((e = hipMalloc(&i8_tmp, (size_t)(2 * max_tpad + 64) * sizeof(float))) != hipSuccess)
      return cleanup_fail(hip_fail(e, "hipMalloc(row scales)"));
    ks = i8_tmp;
    vs = i8_tmp + max_tpad;
    bad = reinterpret_cast<int*>(i8_tmp + 2 * max_tpad);
    if ((e = hipMemsetAsync(bad, 0, sizeof(int), s)) != hipSuccess) return cleanup_fail(hip_fail(e, "hipMemsetAsync"));
  }
  const uint16_t* const* srcs[4] = {pk, rk, pv, rv};
  if (!i8) {
    // every factor one job of pack_batch_kernel, in (block, factor) order; with
    // host sources a batch ends where the staging buffer is full
    const int n_jobs = c->n_blocks * 4;
    std::vector<PackArgs> jobs(n_jobs);
    std::vector<int64_t> starts(n_jobs + 1, 0), stage_at(src_on_device ? 0 : n_jobs);
    std::vector<int> batch_end;
    int64_t fill = 0;
    for (int j = 0; j < n_jobs; ++j) {
      const int b = j / 4, w = j % 4;
      const FactorGeom f = geom_of(*c, b, w);
      const uint16_t* src = srcs[w][b];
      if (!src_on_device) {
        const int64_t elems = round_up((int64_t)f.rows * f.cols, 8);
        if (fill > 0 && fill + elems > stage_elems) {
          batch_end.push_back(j);
          fill = 0;
        }
        stage_at[j] = fill;
        src = staging + fill;
        fill += elems;
      }
      jobs[j] = PackArgs{src, c->data + factor_offset(c->meta[b], w), f, frag_count(f), nullptr};
      starts[j + 1] = starts[j] + frag_count(f);
    }
    batch_end.push_back(n_jobs);
    PackArgs* jobs_d = nullptr;
    const size_t job_bytes = sizeof(PackArgs) * n_jobs, start_bytes = sizeof(int64_t) * (n_jobs + 1);
    if ((e = hipMalloc(&jobs_d, job_bytes + start_bytes)) != hipSuccess)
      return cleanup_fail(hip_fail(e, "hipMalloc(pack jobs)"));
    int64_t* starts_d = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(jobs_d) + job_bytes);
    auto jobs_fail = [&](hipError_t err, const char* what) {
      (void)hipStreamSynchronize(s);
      (void)hipFree(jobs_d);
      return cleanup_fail(hip_fail(err, what));
    };
    if ((e = hipMemcpyAsync(jobs_d, jobs.data(), job_bytes, hipMemcpyHostToDevice, s)) != hipSuccess ||
        (e = hipMemcpyAsync(starts_d, starts.data(), start_bytes, hipMemcpyHostToDevice, s)) != hipSuccess)
      return jobs_fail(e, "hipMemcpyAsync(pack jobs)");
    int j0 = 0;
    for (const int j1 : batch_end) {
      if (!src_on_device)
        for (int j = j0; j < j1; ++j) {
          const FactorGeom& f = jobs[j].geom;
          if ((e = hipMemcpyAsync(staging + stage_at[j], srcs[j % 4][j / 4], (size_t)f.rows * f.cols * 2,
                                  hipMemcpyHostToDevice, s)) != hipSuccess)
            return jobs_fail(e, "hipMemcpyAsync(factor)");
        }
      if ((e = launch_pack_batch(jobs_d + j0, starts_d + j0, j1 - j0, starts[j1] - starts[j0], s)) != hipSuccess)
        return jobs_fail(e, "pack kernel");
      j0 = j1;
    }
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return jobs_fail(e, "hipStreamSynchronize");
    (void)hipFree(jobs_d);
  }
  for (int b = 0; i8 && b < c->n_blocks; ++b) {
    const BlockMeta& m = c->meta[b];
    for (int w = 0; w < 4; ++w) {
      const FactorGeom f = geom_of(*c, b, w);
      const uint16_t* src = srcs[w][b];
      if (!src_on_device) {
        if ((e = hipMemcpyAsync(staging, src, (size_t)f.rows * f.cols * 2, hipMemcpyHostToDevice, s)) != hipSuccess)
          return cleanup_fail(hip_fail(e, "hipMemcpyAsync(factor)"));
        src = staging;
      }
      PackArgs pa{src, c->data + factor_offset(m, w), f, frag_count(f), nullptr};
      if (i8 && (w == kPK || w == kPV)) {
        float* rs = w == kPK ? ks : vs;
        if ((e = launch_row_scales(src, f.rows, f.cols, m.T_pad, rs, bad, s)) != hipSuccess)
          return cleanup_fail(hip_fail(e, "row scale kernel"));
        pa.row_scale = rs;
      }
      if ((e = launch_pack(pa, s)) != hipSuccess) return cleanup_fail(hip_fail(e, "pack kernel"));
    }
    if (i8) {
      float* units = reinterpret_cast<float*>(c->data + i8_scale_offset(m.off_pv, m.T_pad, m.rv_pad));
      if ((e = launch_scale_units(ks, vs, m.T_pad, units, s)) != hipSuccess)
        return cleanup_fail(hip_fail(e, "scale unit kernel"));
    }
  }
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return cleanup_fail(hip_fail(e, "hipStreamSynchronize"));
  if (i8) {
    int flag = 0;
    if ((e = hipMemcpy(&flag, bad, sizeof(int), hipMemcpyDeviceToHost)) != hipSuccess)
      return cleanup_fail(hip_fail(e, "hipMemcpy(flag)"));
    if (flag) return cleanup_fail(fail(MILO_ERR_INVALID_ARG, "a P factor holds a non-finite value (INT8 scales)"));
    (void)hipFree(i8_tmp);
    i8_tmp = nullptr;
  }
  if (staging) (void)hipFree(staging);
  staging = nullptr;
  *out = c;
  return MILO_OK;
}

void milo_cache_free(milo_cache* cache) { destroy(cache); }

int milo_cache_device_bytes(const milo_cache* cache, int64_t* bytes) {
  g_err.clear();
  if (!cache || !bytes) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *bytes = cache->data_elems * 2;
  return MILO_OK;
}

int milo_cache_read_int8(const milo_cache* cache, int32_t block, int32_t which, int8_t* codes, float* scales) {
  g_err.clear();
  if (!cache || !codes || !scales) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  if (!cache->p_int8) return fail(MILO_ERR_INVALID_ARG, "this cache stores bf16 P factors");
  if (block < 0 || block >= cache->n_blocks) return fail(MILO_ERR_INVALID_ARG, "block %d out of range", block);
  if (which != kPK && which != kPV) return fail(MILO_ERR_INVALID_ARG, "which must be 0 (P^K) or 2 (P^V)");
  const BlockMeta& m = cache->meta[block];
  const FactorGeom f = geom_of(*cache, block, which);
  const int64_t nb = i8_factor_bytes(m.T_pad, f.r_pad);
  std::vector<int8_t> packed((size_t)nb);
  MILO_HIP(hipMemcpy(packed.data(), cache->data + factor_offset(m, which), (size_t)nb, hipMemcpyDeviceToHost));
  for (int64_t fr = 0; fr < frag_count(f); ++fr)
    for (int lane = 0; lane < 64; ++lane)
      for (int e = 0; e < 8; ++e) {
        int row, col;
        frag_source(f, fr, lane, e, &row, &col);
        if (row < f.rows && col < f.cols)
          codes[(int64_t)row * f.cols + col] = packed[(size_t)(fr * kFragElems + lane * 8 + e)];
      }
  std::vector<float> units((size_t)i8_scale_bytes(m.T_pad) / 4);
  MILO_HIP(hipMemcpy(units.data(), cache->data + i8_scale_offset(m.off_pv, m.T_pad, m.rv_pad), units.size() * 4,
                     hipMemcpyDeviceToHost));
  for (int t = 0; t < m.T; ++t) scales[t] = units[(size_t)(t / 32) * 64 + (which == kPK ? 0 : 32) + t % 32];
  return MILO_OK;
}

int milo_cache_set_path(milo_cache* cache, int32_t path) {
  g_err.clear();
  if (!cache) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  if (path != MILO_PATH_LATENT && path != MILO_PATH_RECONSTRUCT && path != MILO_PATH_AUTO)
    return fail(MILO_ERR_INVALID_ARG, "path must be MILO_PATH_LATENT, MILO_PATH_RECONSTRUCT or MILO_PATH_AUTO (got %d)",
                path);
  if (cache->p_int8 && path != MILO_PATH_LATENT)
    return fail(MILO_ERR_UNSUPPORTED, "caches with INT8 P factors attend latent only");
  cache->path = path;
  return MILO_OK;
}

int milo_cache_set_rope(milo_cache* cache, double theta, const int64_t* block_pos) {
  g_err.clear();
  if (!cache) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  milo_cache* c = cache;
  if (theta == 0.0) {
    if (!c->rope_pos.empty()) {
      c->rope_pos.clear();
      ++c->rope_gen;
    }
    return MILO_OK;
  }
  if (!std::isfinite(theta) || theta <= 1.0) return fail(MILO_ERR_INVALID_ARG, "theta must be finite and > 1");
  if (c->p_int8) return fail(MILO_ERR_UNSUPPORTED, "caches with INT8 P factors attend latent only");
  // positions: the caller's, or the blocks one after another in id order
  std::vector<int32_t> pos(c->n_blocks);
  int64_t next = 0;
  for (int b = 0; b < c->n_blocks; ++b) {
    const int64_t p = block_pos ? block_pos[b] : next;
    // the padded rows are rotated too (they are zero)
    if (p < 0 || p + c->meta[b].T_pad > kRopeMaxEnd)
      return fail(MILO_ERR_INVALID_ARG, "block %d at position %lld: its %d rows (padded to %d) must lie in [0, %lld)",
                  b, (long long)p, c->T[b], c->meta[b].T_pad, (long long)kRopeMaxEnd);
    pos[b] = (int32_t)p;
    next = p + c->T[b];
  }
  // the frequencies in turns per position, w_j / (2 pi), w_j = theta^(-2j/d)
  const int half = c->d / 2;
  std::vector<double> turns(half);
  for (int j = 0; j < half; ++j) turns[j] = std::pow(theta, -2.0 * j / c->d) / (2.0 * M_PI);
  int dev = -1;
  MILO_HIP(hipGetDevice(&dev));
  if (dev != c->device) return fail(MILO_ERR_INVALID_ARG, "cache lives on device %d, current device is %d", c->device, dev);
  double* t_d = nullptr;
  if (hipMalloc(&t_d, turns.size() * sizeof(double)) != hipSuccess) {
    (void)hipGetLastError();
    return fail(MILO_ERR_OUT_OF_MEMORY, "rotation frequencies");
  }
  if (const hipError_t e = hipMemcpy(t_d, turns.data(), turns.size() * sizeof(double), hipMemcpyHostToDevice);
      e != hipSuccess) {
    (void)hipFree(t_d);
    return hip_fail(e, "rotation frequency upload");
  }
  // earlier calls may still read the old frequencies
  MILO_HIP(hipDeviceSynchronize());
  (void)hipFree(c->rope_d);
  c->rope_d = t_d;
  c->rope_pos = std::move(pos);
  ++c->rope_gen;
  return MILO_OK;
}

int milo_cache_recon_blocks(const milo_cache* cache, int32_t* n) {
  g_err.clear();
  if (!cache || !n) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *n = cache->plan.n_recon_blocks;
  return MILO_OK;
}

int milo_cache_plan_builds(const milo_cache* cache, int64_t* builds) {
  g_err.clear();
  if (!cache || !builds) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  *builds = cache->plan.builds;
  return MILO_OK;
}

int milo_cache_read_factor(const milo_cache* cache, int32_t block, int32_t which, uint16_t* dst) {
  g_err.clear();
  if (!cache || !dst) return fail(MILO_ERR_INVALID_ARG, "NULL argument");
  if (block < 0 || block >= cache->n_blocks) return fail(MILO_ERR_INVALID_ARG, "block %d out of range", block);
  if (which < 0 || which > 3) return fail(MILO_ERR_INVALID_ARG, "which must be 0..3");
  if (cache->p_int8 && (which == kPK || which == kPV))
    return fail(MILO_ERR_INVALID_ARG, "P factors of this cache are stored as INT8 (milo_cache_read_int8)");
  const FactorGeom f = geom_of(*cache, block, which);
  const int64_t n = frag_count(f) * kFragElems;
  std::vector<uint16_t> packed((size_t)n);
  MILO_HIP(hipMemcpy(packed.data(), cache->data + factor_offset(cache->meta[block], which), (size_t)n * 2,
                     hipMemcpyDeviceToHost));
  for (int64_t fr = 0; fr < frag_count(f); ++fr)
    for (int lane = 0; lane < 64; ++lane)
      for (int e = 0; e < 8; ++e) {
        int row, col;
        frag_source(f, fr, lane, e, &row, &col);
        if (row < f.rows && col < f.cols) dst[(int64_t)row * f.cols + col] = packed[(size_t)(fr * kFragElems + lane * 8 + e)];
      }
  return MILO_OK;
}

}  // extern "C"

namespace {

// The workspace a cache owns: device buffers grown on demand (growth waits for
// the stream, since queued calls may still read the old buffers) and a pinned
// staging buffer for plan uploads, rewritten once its previous upload was consumed.
class CacheWorkspace : public Workspace {
 public:
  explicit CacheWorkspace(milo_cache* c) : c_(c) {}
  int upload_plan(const std::vector<unsigned char>& bytes, hipStream_t s, const unsigned char** dev) override {
    milo_cache* c = c_;
    const int64_t plan_bytes = (int64_t)bytes.size();
    if (plan_bytes > c->plan_cap) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->plan_d);
      (void)hipHostFree(c->plan_pinned);
      c->plan_d = nullptr;
      c->plan_pinned = nullptr;
      c->plan_cap = 0;
      c->plan_evt_live = false;
      const int64_t cap = plan_bytes + plan_bytes / 4;
      MILO_HIP(hipMalloc(&c->plan_d, (size_t)cap));
      MILO_HIP(hipHostMalloc(&c->plan_pinned, (size_t)cap, hipHostMallocDefault));
      c->plan_cap = cap;
    }
    if (!c->plan_evt) MILO_HIP(hipEventCreateWithFlags(&c->plan_evt, hipEventDisableTiming));
    if (c->plan_evt_live) MILO_HIP(hipEventSynchronize(c->plan_evt));
    c->plan_evt_live = false;
    std::memcpy(c->plan_pinned, bytes.data(), (size_t)plan_bytes);
    MILO_HIP(hipMemcpyAsync(c->plan_d, c->plan_pinned, (size_t)plan_bytes, hipMemcpyHostToDevice, s));
    MILO_HIP(hipEventRecord(c->plan_evt, s));
    c->plan_evt_live = true;
    *dev = c->plan_d;
    return MILO_OK;
  }
  int partials(int64_t need, int d, hipStream_t s, float** o, float2** ml) override {
    milo_cache* c = c_;
    if (need > c->part_cols_slots) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->part_o);
      (void)hipFree(c->part_ml);
      c->part_o = nullptr;
      c->part_ml = nullptr;
      c->part_cols_slots = 0;
      const int64_t cap = env_byte_cap();
      const int64_t bytes = need * ((int64_t)d * 4 + 8);
      if (cap >= 0 && c->data_elems * 2 + bytes > cap)
        return fail(MILO_ERR_OUT_OF_MEMORY, "workspace of %lld bytes exceeds MILO_MAX_DEVICE_BYTES",
                    (long long)bytes);
      MILO_HIP(hipMalloc(&c->part_o, (size_t)need * d * 4));
      MILO_HIP(hipMalloc(&c->part_ml, (size_t)need * sizeof(float2)));
      c->part_cols_slots = need;
    }
    *o = c->part_o;
    *ml = c->part_ml;
    return MILO_OK;
  }
  int tail_lengths(const int32_t* host, int n_q, hipStream_t s, const int32_t** dev) override {
    milo_cache* c = c_;
    if (n_q > c->tail_len_cap) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->tail_len_d);
      c->tail_len_d = nullptr;
      c->tail_len_cap = 0;
      MILO_HIP(hipMalloc(&c->tail_len_d, sizeof(int32_t) * n_q));
      c->tail_len_cap = n_q;
    }
    MILO_HIP(hipMemcpyAsync(c->tail_len_d, host, sizeof(int32_t) * n_q, hipMemcpyHostToDevice, s));
    *dev = c->tail_len_d;
    return MILO_OK;
  }
  bool may_time() const override { return true; }
  bool can_recon() const override { return true; }
  int recon_buffer(int64_t elems, const uint16_t* data, hipStream_t s, uint16_t** buf) override {
    milo_cache* c = c_;
    if (elems > c->recon_cap) {
      MILO_HIP(hipStreamSynchronize(s));
      (void)hipFree(c->recon_raw);
      c->recon_raw = nullptr;
      c->recon_d = nullptr;
      c->recon_cap = 0;
      const int64_t cap = env_byte_cap();
      const int64_t bytes = elems * 2 + 1024;
      if (cap >= 0 && c->data_elems * 2 + bytes > cap)
        return fail(MILO_ERR_OUT_OF_MEMORY, "reconstruction buffer of %lld bytes exceeds MILO_MAX_DEVICE_BYTES",
                    (long long)bytes);
      MILO_HIP(hipMalloc(&c->recon_raw, (size_t)bytes));
      // start a whole number of 1 KiB fragments from the factor buffer
      const uintptr_t raw = reinterpret_cast<uintptr_t>(c->recon_raw), base = reinterpret_cast<uintptr_t>(data);
      const uintptr_t adj = (base - raw) & 1023u;
      c->recon_d = reinterpret_cast<uint16_t*>(c->recon_raw + adj);
      c->recon_cap = elems;
    }
    *buf = c->recon_d;
    return MILO_OK;
  }

 private:
  milo_cache* c_;
};

// Reconstruct-then-attend pays for a block when rebuilding its keys and values
// and attending them densely is clearly faster than the latent route.  Per-block
// times (microseconds) fitted to MI355X kernel timings of the 7B- (28-layer) and
// 14B-shaped steps, for a block of T tokens, ranks rk / rv, N query columns,
// D = H_kv d:
//   latent        4.24e-9 N (rk + rv)(T + d)        (latent block items)
//   reconstruct   4.17e-9 T D (rk + rv)             (reconstruction GEMMs)
//               + 1.99e-6 T D                       (writing, then reading, the 16-bit K and V)
//               + 7.06e-9 N T d                     (dense block items)
// and reconstruction is chosen below 0.85 of the latent time (mixed plans
// measured slower than the sum of their parts near the tie).
bool recon_pays(int T, int rk, int rv, int64_t N, int D, int d) {
  const double r = (double)rk + rv;
  const double lat = 4.24e-9 * (double)N * r * (T + d);
  const double rec = 4.17e-9 * (double)T * D * r + 1.99e-6 * (double)T * D + 7.06e-9 * (double)N * T * d;
  return rec < 0.85 * lat;
}

}  // namespace

namespace milo {

int attend_call(milo_cache* c, PlanState& ps, Workspace& ws, const int32_t* block_table, int32_t n_sel, int32_t n_q,
                int32_t n_q_heads, const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v,
                const int32_t* tail_len, int32_t tail_base, int32_t tail_cap, int64_t tail_stride, float scale,
                float* out, void* hip_stream) {
  // ---- validation (host only, nothing queued yet) ----
  if (!c) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  if (n_sel < 0) return fail(MILO_ERR_INVALID_ARG, "n_sel must be >= 0");
  if (n_sel > 0 && !block_table) return fail(MILO_ERR_INVALID_ARG, "block_table is NULL");
  if (n_q < 1) return fail(MILO_ERR_INVALID_ARG, "n_q must be >= 1");
  if (n_q_heads < 1 || n_q_heads % c->n_kv != 0)
    return fail(MILO_ERR_INVALID_ARG, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)", n_q_heads,
                c->n_kv);
  const int G = n_q_heads / c->n_kv;
  if (G > kMaxGroup) return fail(MILO_ERR_UNSUPPORTED, "more than %d query heads per KV head", kMaxGroup);
  if (!q || !out) return fail(MILO_ERR_INVALID_ARG, "q / out must be non-NULL");
  if (tail_cap < 0) return fail(MILO_ERR_INVALID_ARG, "tail_cap must be >= 0");
  const bool causal = tail_len == nullptr && tail_base >= 0;
  if (tail_cap > 0 && (!tail_k || !tail_v || (!tail_len && !causal)))
    return fail(MILO_ERR_INVALID_ARG, "tail_k / tail_v / tail_len must be non-NULL when tail_cap > 0");
  if (!std::isfinite(scale)) return fail(MILO_ERR_INVALID_ARG, "scale must be finite");
  if ((int64_t)n_q * n_q_heads > (int64_t)1 << 24) return fail(MILO_ERR_UNSUPPORTED, "too many query columns");
  int max_len = 0;
  for (int i = 0; i < n_q; ++i) {
    const int len = causal ? tail_base + i + 1 : tail_cap > 0 ? tail_len[i] : 0;
    if (len < 0 || len > tail_cap)
      return fail(MILO_ERR_INVALID_ARG, "tail_len[%d]=%d outside [0, tail_cap=%d]", i, len, tail_cap);
    if (n_sel == 0 && len == 0) return fail(MILO_ERR_INVALID_ARG, "request %d has no keys to attend to", i);
    max_len = std::max(max_len, len);
  }
  if (n_sel > 0) {
    std::vector<char> seen(c->n_blocks, 0);
    for (int j = 0; j < n_sel; ++j) {
      const int b = block_table[j];
      if (b < 0 || b >= c->n_blocks)
        return fail(MILO_ERR_INVALID_ARG, "block_table[%d]=%d outside [0, %d)", j, b, c->n_blocks);
      if (seen[b]) return fail(MILO_ERR_INVALID_ARG, "block id %d selected twice", b);
      seen[b] = 1;
    }
  }
  int dev = -1;
  MILO_HIP(hipGetDevice(&dev));
  if (dev != c->device) return fail(MILO_ERR_INVALID_ARG, "cache lives on device %d, current device is %d", c->device, dev);
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);

  // ---- which blocks are reconstructed (milo_cache_set_path; every block of a
  // cache with pre-RoPE keys, milo_cache_set_rope) ----
  const bool rope = !c->rope_pos.empty();
  if ((c->path == MILO_PATH_RECONSTRUCT || (rope && n_sel > 0)) && !ws.can_recon())
    return fail(MILO_ERR_UNSUPPORTED, "this entry point attends latent only (reconstruction needs a workspace)");
  std::vector<char> recon((size_t)std::max(n_sel, 1), 0);
  int n_recon = 0;
  for (int j = 0; j < n_sel; ++j) {
    const int b = block_table[j];
    // ranks beyond the latent route's reach are always reconstructed
    const bool must = c->rk[b] > kMaxRank || c->rv[b] > kMaxRank;
    if (must && !ws.can_recon())
      return fail(MILO_ERR_UNSUPPORTED, "block %d has rank above %d and needs reconstruction, which this entry point "
                  "does not do", b, kMaxRank);
    if (must || rope) recon[j] = 1;
    else if (c->path != MILO_PATH_LATENT && ws.can_recon())
      recon[j] = c->path == MILO_PATH_RECONSTRUCT ||
                 recon_pays(c->T[b], c->rk[b], c->rv[b], (int64_t)n_q * n_q_heads, c->n_kv * c->d, c->d);
    n_recon += recon[j];
  }

  // ---- the latent projection: MFMA (measured faster on gfx950 at every batch,
  // 7 columns per KV head included), or a wavefront GEMV kernel variant for
  // small batches (at most kGemvCols query columns per KV head, bf16 P factors)
  // when the MILO_PROJECTION environment variable says "gemv" ----
  const int N_g = n_q * G;
  bool gemv = false;
  if (const char* pe = std::getenv("MILO_PROJECTION"); pe && *pe) {
    if (std::strcmp(pe, "gemv") == 0) {
      if (N_g > kGemvCols || c->p_int8)
        return fail(MILO_ERR_UNSUPPORTED,
                    "the GEMV projection needs bf16 P factors and at most %d query columns per KV head (got %d)",
                    kGemvCols, N_g);
      gemv = true;
    } else if (std::strcmp(pe, "mfma") != 0) {
      return fail(MILO_ERR_INVALID_ARG, "MILO_PROJECTION must be mfma or gemv (got %s)", pe);
    }
  }

  // ---- a prefill chunk of kSharedTailMinTokens tokens or more attends its
  // shared tail once per KV head: packed like a reconstructed block (rows up to
  // a planned capacity, the longest tail rounded up to a power of two of
  // 256-token tiles, at most tail_cap) and read by dense items whose columns
  // mask tokens past their causal limit.  Smaller chunks (measured on the
  // 7B-shaped layer after 256 tail rows: 16 tokens +16%, 64 tokens +3%, 256
  // tokens -5% attention time with the packed tail), INT8 caches and
  // workspaces without a reconstruction buffer use tail items per token ----
  constexpr int kSharedTailMinTokens = 128;
  const bool shared_tail =
      causal && max_len > 0 && n_q >= kSharedTailMinTokens && !c->p_int8 && ws.can_recon();
  int tail_tiles = 0;
  if (shared_tail) {
    tail_tiles = 1;
    while (tail_tiles * kTile < max_len) tail_tiles *= 2;
    tail_tiles = std::min(tail_tiles, (tail_cap + kTile - 1) / kTile);
  }

  // ---- plan: rebuilt only when the block table, the batch shape or the tail
  // chunk capacity changes (the longest tail rounded up to a power of two of
  // chunks, at most tail_cap), not when tails merely grow ----
  const int need_chunks = shared_tail ? 0 : (max_len + kTailChunk - 1) / kTailChunk;
  int n_chunks = 0;
  if (need_chunks > 0) {
    n_chunks = 1;
    while (n_chunks < need_chunks) n_chunks *= 2;
    n_chunks = std::min(n_chunks, (tail_cap + kTailChunk - 1) / kTailChunk);
  }
  std::vector<int32_t> key;
  key.reserve(6 + n_sel);
  key.push_back((int32_t)(c->serial & 0xffffffffu));  // the cache (plans of a shared workspace)
  key.push_back((int32_t)(c->serial >> 32));
  key.push_back(n_sel);
  key.push_back(n_q);
  key.push_back(n_q_heads);
  key.push_back(n_chunks);
  key.push_back(n_recon > 0 ? c->path : MILO_PATH_LATENT);
  key.push_back(n_recon);
  key.push_back(gemv ? 1 : 0);
  key.push_back(tail_tiles);
  key.push_back(rope ? c->rope_gen : -1);
  key.insert(key.end(), block_table, block_table + n_sel);
  const int n_cols = n_q * n_q_heads;
  if (key != ps.key) {
    // no plan is valid until this one is complete: a failure below (an
    // allocation, an upload) must not leave the old key pointing at buffers
    // that were freed or half rewritten
    ps.key.clear();
    std::vector<int64_t> region;
    ReconPlan rp;
    // the blocks the plan sees: the cache's, plus the packed shared tail as
    // block n_blocks after the table's last entry
    std::vector<BlockMeta> meta_x;
    std::vector<int32_t> table_x(block_table, block_table + n_sel);
    int64_t tail_region = -1;
    if (n_recon > 0 || shared_tail) {
      region.assign(c->n_blocks + 1, -1);
      build_recon_plan(c->meta.data(), block_table, n_sel, recon.data(), c->n_kv, c->d, &region, &rp,
                       rope ? c->rope_pos.data() : nullptr);
    }
    if (shared_tail) {
      meta_x = c->meta;
      BlockMeta tm{};
      tm.T = tail_tiles * kTile;
      tm.T_pad = tail_tiles * kTile;
      tm.rk_pad = tm.rv_pad = c->d;
      meta_x.push_back(tm);
      tail_region = rp.elems;
      region[c->n_blocks] = tail_region;
      rp.elems += 2LL * tm.T_pad * c->n_kv * c->d;
      table_x.push_back(c->n_blocks);
    }
    const Tiling til = make_tiling(c->n_kv, n_q * G, n_recon > 0 || shared_tail, gemv ? kGemvCols : kCols);
    Schedule sch;
    std::string why;
    PlanInput pin{shared_tail ? meta_x.data() : c->meta.data(), c->n_kv, c->d, c->p_int8};
    pin.recon_region = region.empty() ? nullptr : region.data();
    pin.causal_block = shared_tail ? c->n_blocks : -1;
    if (!build_schedule(pin, table_x.data(), (int)table_x.size(), n_q, n_chunks, til, env_program_cap(), &sch, &why))
      return fail(MILO_ERR_UNSUPPORTED, "%s", why.c_str());
    // the reconstruction table and tasks follow the schedule in the plan
    int64_t rb_off = 0, rt_off = 0;
    if (n_recon > 0) {
      rb_off = (int64_t)round_up((int64_t)sch.bytes.size(), 64);
      rt_off = rb_off + (int64_t)(rp.blocks.size() * sizeof(ReconBlock));
      sch.bytes.resize((size_t)(rt_off + (int64_t)(rp.tasks.size() * sizeof(int2))));
      std::memcpy(sch.bytes.data() + rb_off, rp.blocks.data(), rp.blocks.size() * sizeof(ReconBlock));
      std::memcpy(sch.bytes.data() + rt_off, rp.tasks.data(), rp.tasks.size() * sizeof(int2));
    }
    const int max_rt = sch.max_own <= 2 ? 2 : sch.max_own == 3 ? 3 : 4;
    // deepest fragment ring that fits next to the program, projected query and
    // weight tile (4 slots go with the half weight tile)
    const size_t base = attend_lds_base_bytes(c->d, sch.rk_pad_max, sch.rv_pad_max, sch.half_w);
    const size_t prog = (size_t)sch.prog_bytes;
    int nslot = 0;
    if (sch.half_w) {
      // the program was sized to leave room for this ring
      if (prog + base + attend_ring_bytes(4) > (size_t)kLdsBytes)
        return fail(MILO_ERR_UNSUPPORTED, "work schedule does not fit in LDS");
      nslot = 4;
    } else {
      for (int cand : {8, 6})
        if (prog + base + attend_ring_bytes(cand) <= (size_t)kLdsBytes) { nslot = cand; break; }
    }
    // the workspace for the new plan's partials first (a workspace that cannot
    // hold them fails here, before anything is queued), then the upload, in
    // stream order: the kernels of earlier calls, queued before the copy, read
    // the old plan first
    float* po = nullptr;
    float2* pml = nullptr;
    if (const int err = ws.partials((int64_t)n_cols * (sch.n_block_slots + n_chunks), c->d, s, &po, &pml);
        err != MILO_OK)
      return err;
    const unsigned char* plan_d = nullptr;
    if (const int err = ws.upload_plan(sch.bytes, s, &plan_d); err != MILO_OK) return err;
    ps.plan_d = plan_d;
    ps.n_launch = sch.n_launch;
    ps.n_chunks = n_chunks;
    ps.n_slots = sch.n_block_slots + n_chunks;
    ps.n_block_slots = sch.n_block_slots;
    ps.count_off = sch.count_off;
    ps.tiles = til.geom;
    ps.max_rt = max_rt;
    ps.nslot = nslot;
    ps.rk_pad_max = sch.rk_pad_max;
    ps.prog_bytes = sch.prog_bytes;
    ps.ring_offset = (int)base;
    ps.lds = prog + base + attend_ring_bytes(nslot);
    ps.n_recon_blocks = (int)rp.blocks.size();
    ps.n_recon_tasks = (int)rp.tasks.size();
    ps.recon_blocks_off = rb_off;
    ps.recon_tasks_off = rt_off;
    ps.recon_elems = rp.elems;
    ps.tail_region = tail_region;
    ps.run_cap = sch.run_cap;
    ps.tail_T_pad = tail_tiles * kTile;
    ps.gemv = gemv;
    ps.key.swap(key);
    ++ps.builds;
  }
  float* part_o = nullptr;
  float2* part_ml = nullptr;
  if (const int err = ws.partials((int64_t)n_cols * ps.n_slots, c->d, s, &part_o, &part_ml); err != MILO_OK)
    return err;
  // this call's tail lengths travel in the kernel arguments; a batch above
  // kInlineTails requests copies them to the device in stream order
  TailLens tls{};
  if (causal || tail_cap == 0) {
    tls.mode = kTailAffine;
    tls.base = causal ? tail_base + 1 : 0;
    tls.step = causal ? 1 : 0;
  } else if (n_q <= kInlineTails) {
    tls.mode = kTailInline;
    for (int i = 0; i < n_q; ++i) tls.v[i] = tail_len[i];
  } else {
    tls.mode = kTailDevice;
    if (const int err = ws.tail_lengths(tail_len, n_q, s, &tls.dev); err != MILO_OK) return err;
  }

  // reconstruction buffer of this call
  uint16_t* rbuf = nullptr;
  int recon_delta = 0;
  if (ps.recon_elems > 0) {
    if (const int err = ws.recon_buffer(ps.recon_elems, c->data, s, &rbuf); err != MILO_OK) return err;
    const int64_t dbytes = (reinterpret_cast<const unsigned char*>(rbuf) - reinterpret_cast<const unsigned char*>(c->data));
    const int64_t dfr = dbytes / (kFragElems * 2);
    if (dbytes % (kFragElems * 2) != 0 || dfr < -((int64_t)1 << 30) || dfr + ps.recon_elems / kFragElems > ((int64_t)1 << 30))
      return fail(MILO_ERR_UNSUPPORTED, "reconstruction buffer out of the fragment index range of the factor buffer");
    recon_delta = (int)dfr;
  }

  // ---- launches ----
  AttendArgs aa{};
  aa.data = c->data;
  aa.recon_delta = recon_delta;
  aa.run_cap = ps.run_cap;
  aa.prog = ps.plan_d;
  aa.q = q;
  aa.tail_k = tail_k;
  aa.tail_v = tail_v;
  aa.part_o = part_o;
  aa.part_ml = part_ml;
  aa.qscale = scale * 1.4426950408889634f;
  aa.n_q = n_q;
  aa.H_q = n_q_heads;
  aa.H_kv = c->n_kv;
  aa.G = G;
  aa.tail_stride = tail_stride;
  aa.n_slots = ps.n_slots;
  aa.n_block_slots = ps.n_block_slots;
  aa.qt_stride = ps.rk_pad_max + 8;
  aa.prog_bytes = ps.prog_bytes;
  aa.ring_offset = ps.ring_offset;
  aa.N_g = n_q * G;
  aa.tl = tls;
  MergeArgs ma{};
  ma.part_o = part_o;
  ma.part_ml = part_ml;
  ma.out = out;
  ma.slot_count = reinterpret_cast<const int32_t*>(ps.plan_d + ps.count_off);
  ma.H_q = n_q_heads;
  ma.G = G;
  ma.n_block_slots = ps.n_block_slots;
  ma.n_slots = ps.n_slots;
  ma.tiles = ps.tiles;
  ma.tl = tls;
  if (ps.tail_region >= 0) {  // the shared tail's partials sit in block slots
    ma.tl = TailLens{};
    ma.tl.mode = kTailAffine;
  }

  // timing: events recorded by the launches themselves at kernel start and end
  // attend start / end, merge start / end, reconstruction start / end
  hipEvent_t ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  const int n_ev = ps.n_recon_tasks > 0 ? 6 : 4;
  bool timed = false;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    if (g_timing.enabled && ws.may_time()) {
      for (int k = 0; k < n_ev; ++k) {
        if (g_timing.pool.empty()) {
          hipEvent_t e;
          const hipError_t ce = hipEventCreate(&e);
          if (ce != hipSuccess) {
            for (int j = 0; j < k; ++j) g_timing.pool.push_back(ev[j]);
            return hip_fail(ce, "hipEventCreate");
          }
          g_timing.pool.push_back(e);
        }
        ev[k] = g_timing.pool.back();
        g_timing.pool.pop_back();
      }
      timed = true;
    }
  }
  // a failed launch hands the call's events back to the pool
  auto launch_fail = [&](hipError_t err, const char* what) {
    if (timed) {
      std::lock_guard<std::mutex> lk(g_timing.mu);
      g_timing.pool.insert(g_timing.pool.end(), ev, ev + n_ev);
    }
    return hip_fail(err, what);
  };
  hipError_t e = hipSuccess;
  if (ps.n_recon_tasks > 0) {
    ReconArgs ra{};
    ra.data = c->data;
    ra.recon = rbuf;
    ra.blocks = reinterpret_cast<const ReconBlock*>(ps.plan_d + ps.recon_blocks_off);
    ra.tasks = reinterpret_cast<const int2*>(ps.plan_d + ps.recon_tasks_off);
    ra.rope_turns = c->rope_d;
    e = launch_recon(ra, c->d, ps.n_recon_tasks, s, ev[4], ev[5]);
    if (e != hipSuccess) return launch_fail(e, "reconstruction kernel launch");
  }
  if (ps.tail_region >= 0) {
    TailPackArgs ta{};
    ta.tail_k = tail_k;
    ta.tail_v = tail_v;
    ta.recon = rbuf;
    ta.region = ps.tail_region;
    ta.rows = max_len;
    ta.T_pad = ps.tail_T_pad;
    ta.n_kv = c->n_kv;
    e = launch_pack_tail(ta, c->d, s);
    if (e != hipSuccess) return launch_fail(e, "tail packing kernel launch");
  }
  for (int l = 0; l < ps.n_launch; ++l) {
    aa.wg = reinterpret_cast<const WgProgram*>(ps.plan_d) + (size_t)l * kCUs;
    e = launch_attend(aa, c->d, ps.max_rt, ps.nslot, c->p_int8, ps.gemv, kCUs, ps.lds, s, l == 0 ? ev[0] : nullptr,
                      l == ps.n_launch - 1 ? ev[1] : nullptr);
    if (e != hipSuccess) return launch_fail(e, "attend kernel launch");
  }
  e = launch_merge(ma, c->d, n_cols, s, ev[2], ev[3]);
  if (e != hipSuccess) return launch_fail(e, "merge kernel launch");
  if (timed) {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    g_timing.recorded.insert(g_timing.recorded.end(), ev, ev + 4);
    if (n_ev == 6) g_timing.recon_recorded.insert(g_timing.recon_recorded.end(), ev + 4, ev + 6);
  }
  return MILO_OK;
}

}  // namespace milo

extern "C" {

int milo_attend_decode(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_q, int32_t n_q_heads,
                       const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v, const int32_t* tail_len,
                       int32_t tail_cap, float scale, float* out, void* hip_stream) {
  g_err.clear();
  if (!c) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  if (tail_cap > 0 && !tail_len) return fail(MILO_ERR_INVALID_ARG, "tail_len must be non-NULL when tail_cap > 0");
  CacheWorkspace ws(c);
  return attend_call(c, c->plan, ws, block_table, n_sel, n_q, n_q_heads, q, tail_k, tail_v, tail_len, -1, tail_cap,
                     tail_cap, scale, out, hip_stream);
}

int milo_attend_prefill(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_tok, int32_t n_q_heads,
                        const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v, int32_t tail_base,
                        int32_t tail_cap, float scale, float* out, void* hip_stream) {
  g_err.clear();
  if (n_tok < 1) return fail(MILO_ERR_INVALID_ARG, "n_tok must be >= 1");
  if (tail_base < 0) return fail(MILO_ERR_INVALID_ARG, "tail_base must be >= 0");
  if ((int64_t)tail_base + n_tok > tail_cap)
    return fail(MILO_ERR_INVALID_ARG, "tail_cap (%d) must hold tail_base + n_tok = %lld rows", tail_cap,
                (long long)tail_base + n_tok);
  if (!tail_k || !tail_v) return fail(MILO_ERR_INVALID_ARG, "tail_k / tail_v must be non-NULL");
  if (!c) return fail(MILO_ERR_INVALID_ARG, "cache is NULL");
  // token j sees the tail_base rows before the chunk and the chunk's first j + 1 tokens
  CacheWorkspace ws(c);
  return attend_call(c, c->plan, ws, block_table, n_sel, n_tok, n_q_heads, q, tail_k, tail_v, nullptr, tail_base,
                     tail_cap, 0, scale, out, hip_stream);
}

int milo_timing_enable(int enable) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.enabled = enable != 0;
  return MILO_OK;
}

int milo_timing_read_recon(double* recon_kernel_ms, int64_t* n_calls) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double t = 0.0;
  const size_t n = g_timing.recon_recorded.size() / 2;
  for (size_t k = 0; k < n; ++k) {
    hipEvent_t* e = &g_timing.recon_recorded[2 * k];
    MILO_HIP(hipEventSynchronize(e[1]));
    float ms = 0.f;
    MILO_HIP(hipEventElapsedTime(&ms, e[0], e[1]));
    t += ms;
  }
  g_timing.pool.insert(g_timing.pool.end(), g_timing.recon_recorded.begin(), g_timing.recon_recorded.end());
  g_timing.recon_recorded.clear();
  if (recon_kernel_ms) *recon_kernel_ms = t;
  if (n_calls) *n_calls = (int64_t)n;
  return MILO_OK;
}

int milo_timing_read(double* attend_kernel_ms, double* merge_kernel_ms, int64_t* n_calls) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double ta = 0.0, tm = 0.0;
  const size_t n = g_timing.recorded.size() / 4;
  for (size_t k = 0; k < n; ++k) {
    hipEvent_t* e = &g_timing.recorded[4 * k];
    MILO_HIP(hipEventSynchronize(e[3]));
    float a = 0.f, m = 0.f;
    MILO_HIP(hipEventElapsedTime(&a, e[0], e[1]));
    MILO_HIP(hipEventElapsedTime(&m, e[2], e[3]));
    ta += a;
    tm += m;
  }
  g_timing.pool.insert(g_timing.pool.end(), g_timing.recorded.begin(), g_timing.recorded.end());
  g_timing.recorded.clear();
  if (attend_kernel_ms) *attend_kernel_ms = ta;
  if (merge_kernel_ms) *merge_kernel_ms = tm;
  if (n_calls) *n_calls = (int64_t)n;
  return MILO_OK;
}


}  // extern "C"
