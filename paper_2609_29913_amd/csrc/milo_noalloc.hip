// The attention entry point that allocates nothing: milo_attend_decode with its
// workspace (the work plan, the partial results, the tail lengths of large
// batches) in a fixed scratch array of the library instead of device memory
// the cache allocates and grows.  For callers that cannot allocate: code under
// HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "milo.h"
#include "milo_attend.h"
#include "milo_internal.h"

namespace milo {
namespace {

// Scratch layout (bytes): [0, 8 MiB) the work plan; [8 MiB, 9 MiB) the tail
// lengths of batches above kInlineTails requests; [9 MiB, 64 MiB) the partial
// results, per-column (max, sum) pairs then 256-byte aligned partial outputs.
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr size_t kScratchPlanBytes = (size_t)8 << 20;
constexpr size_t kScratchTailOff = kScratchPlanBytes;
constexpr size_t kScratchTailBytes = (size_t)1 << 20;
constexpr size_t kScratchPartOff = kScratchTailOff + kScratchTailBytes;
constexpr int kMaxDevices = 64;

// One copy per GPU the library runs on, held until the process ends.  In host
// code this name is a host-side stand-in, not a device address: the device
// address of each GPU's copy comes from hipGetSymbolAddress (DeviceScratch::ptr).
__device__ __align__(256) unsigned char scratch[kScratchBytes];

struct DeviceScratch {
  std::mutex mu;                          // one call at a time per GPU on the host side
  unsigned char* ptr = nullptr;           // this GPU's scratch (hipGetSymbolAddress, once)
  PlanState plan;                         // the plan the scratch holds
  std::vector<unsigned char> host_plan;   // source of the last plan upload
};
DeviceScratch g_dev[kMaxDevices];

int scratch_fail(int code, const char* fmt, long long a, long long b) {
  char buf[256];
  std::snprintf(buf, sizeof buf, fmt, a, b);
  return report_error(code, buf);
}

// The workspace of the scratch array: fixed regions, checked against their
// limits; nothing is allocated on the device.
class ScratchWorkspace : public Workspace {
 public:
  explicit ScratchWorkspace(DeviceScratch& d) : d_(d) {}
  int upload_plan(const std::vector<unsigned char>& bytes, hipStream_t s, const unsigned char** dev) override {
    if (bytes.size() > kScratchPlanBytes)
      return scratch_fail(MILO_ERR_UNSUPPORTED, "work plan of %lld bytes exceeds the scratch's %lld-byte plan region",
                          (long long)bytes.size(), (long long)kScratchPlanBytes);
    d_.host_plan = bytes;
    const hipError_t e =
        hipMemcpyAsync(d_.ptr, d_.host_plan.data(), d_.host_plan.size(), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return report_error(MILO_ERR_HIP, hipGetErrorString(e));
    *dev = d_.ptr;
    return MILO_OK;
  }
  int partials(int64_t cols_slots, int d, hipStream_t, float** o, float2** ml) override {
    const size_t ml_bytes = ((size_t)cols_slots * sizeof(float2) + 255) / 256 * 256;
    const size_t need = ml_bytes + (size_t)cols_slots * d * 4;
    if (need > kScratchBytes - kScratchPartOff)
      return scratch_fail(MILO_ERR_UNSUPPORTED,
                          "partial results of %lld bytes exceed the scratch's %lld-byte region "
                          "(use milo_attend_decode, which grows its own workspace)",
                          (long long)need, (long long)(kScratchBytes - kScratchPartOff));
    *ml = reinterpret_cast<float2*>(d_.ptr + kScratchPartOff);
    *o = reinterpret_cast<float*>(d_.ptr + kScratchPartOff + ml_bytes);
    return MILO_OK;
  }
  int tail_lengths(const int32_t* host, int n_q, hipStream_t s, const int32_t** dev) override {
    if ((size_t)n_q * sizeof(int32_t) > kScratchTailBytes)
      return scratch_fail(MILO_ERR_UNSUPPORTED, "%lld tail lengths exceed the scratch's room for %lld",
                          (long long)n_q, (long long)(kScratchTailBytes / sizeof(int32_t)));
    int32_t* dst = reinterpret_cast<int32_t*>(d_.ptr + kScratchTailOff);
    const hipError_t e = hipMemcpyAsync(dst, host, sizeof(int32_t) * n_q, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return report_error(MILO_ERR_HIP, hipGetErrorString(e));
    *dev = dst;
    return MILO_OK;
  }
  bool may_time() const override { return false; }

 private:
  DeviceScratch& d_;
};

}  // namespace
}  // namespace milo

using namespace milo;

extern "C" int milo_attend_decode_noalloc(milo_cache* c, const int32_t* block_table, int32_t n_sel, int32_t n_q,
                                          int32_t n_q_heads, const uint16_t* q, const uint16_t* tail_k,
                                          const uint16_t* tail_v, const int32_t* tail_len, int32_t tail_cap,
                                          float scale, float* out, void* hip_stream) {
  clear_error();
  if (!c) return report_error(MILO_ERR_INVALID_ARG, "cache is NULL");
  if (tail_cap > 0 && !tail_len) return report_error(MILO_ERR_INVALID_ARG, "tail_len must be non-NULL when tail_cap > 0");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return report_error(MILO_ERR_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return report_error(MILO_ERR_UNSUPPORTED, "device index out of range");
  DeviceScratch& d = g_dev[dev];
  std::lock_guard<std::mutex> lk(d.mu);
  if (!d.ptr) {
    // first call on this device (it is current): the device address of its copy
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return report_error(MILO_ERR_HIP, "hipGetSymbolAddress(scratch) failed");
    d.ptr = static_cast<unsigned char*>(p);
  }
  ScratchWorkspace ws(d);
  return attend_call(c, d.plan, ws, block_table, n_sel, n_q, n_q_heads, q, tail_k, tail_v, tail_len, -1, tail_cap,
                     tail_cap, scale, out, hip_stream);
}
