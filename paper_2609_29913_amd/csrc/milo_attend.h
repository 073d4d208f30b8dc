// One attention call (host side), shared by the entry points that own their
// workspace (milo_attend_decode / milo_attend_prefill: device memory of the
// cache, grown on demand) and the one that allocates nothing
// (milo_attend_decode_noalloc: a fixed scratch region of the library).
#pragma once

#include <stdint.h>

#include <vector>

#include "milo.h"
#include "milo_internal.h"

struct milo_cache;

namespace milo {

// The work plan of the last call shape attended through one workspace, and the
// launch parameters that go with it.
struct PlanState {
  std::vector<int32_t> key;  // call shape the plan was built for (empty: none)
  int64_t builds = 0;
  const unsigned char* plan_d = nullptr;  // device copy of the plan
  int n_launch = 0, n_slots = 0, n_block_slots = 0, max_rt = 0, nslot = 0, rk_pad_max = 0, n_chunks = 0;
  TileGeom tiles{};
  int64_t count_off = 0;  // byte offset of the plan's slot counts
  int prog_bytes = 0, ring_offset = 0;
  size_t lds = 0;
  // reconstruct-then-attend: reconstructed blocks, their table and tasks in the plan
  int n_recon_blocks = 0, n_recon_tasks = 0;
  int64_t recon_blocks_off = 0, recon_tasks_off = 0;  // byte offsets in the plan
  int64_t recon_elems = 0;                            // reconstruction buffer (bf16 elements)
  bool gemv = false;                                  // latent projection as a wavefront GEMV
  int run_cap = kRunCap;                              // run buffer entries of the plan
  int64_t tail_region = -1;                           // a prefill chunk's packed shared tail (or -1)
  int tail_T_pad = 0;                                 // its planned rows
};

// Device memory one attention call uses beyond its inputs and outputs.  Each
// method returns MILO_OK or an error code with the calling thread's message set.
class Workspace {
 public:
  virtual ~Workspace() = default;
  // queue the upload of a plan in stream order; *dev receives its device address
  virtual int upload_plan(const std::vector<unsigned char>& bytes, hipStream_t s, const unsigned char** dev) = 0;
  // partial results for cols_slots (column, slot) pairs of head dimension d
  virtual int partials(int64_t cols_slots, int d, hipStream_t s, float** o, float2** ml) = 0;
  // device copy of n_q tail lengths (batches above kInlineTails), queued in stream order
  virtual int tail_lengths(const int32_t* host, int n_q, hipStream_t s, const int32_t** dev) = 0;
  // whether the call may take timing events from the library's pool (creating some when it is empty)
  virtual bool may_time() const = 0;
  // reconstruct-then-attend: a buffer of `elems` bf16 elements whose distance
  // from `data` is a whole number of 1 KiB fragments; workspaces that cannot
  // hold one return false from can_recon (their calls attend every block latent)
  virtual bool can_recon() const { return false; }
  virtual int recon_buffer(int64_t elems, const uint16_t* data, hipStream_t s, uint16_t** buf) {
    (void)elems; (void)data; (void)s; (void)buf;
    return MILO_ERR_UNSUPPORTED;
  }
};

// Attention of n_q query tokens over the selected blocks plus their dense tails
// (see milo_attend_decode): query i reads tail rows [i * tail_stride,
// i * tail_stride + len_i) of tail_k / tail_v with len_i = tail_len[i] (host
// array), or tail_base + i + 1 when tail_len is NULL (a prefill chunk).
int attend_call(milo_cache* c, PlanState& ps, Workspace& ws, const int32_t* block_table, int32_t n_sel, int32_t n_q,
                int32_t n_q_heads, const uint16_t* q, const uint16_t* tail_k, const uint16_t* tail_v,
                const int32_t* tail_len, int32_t tail_base, int32_t tail_cap, int64_t tail_stride, float scale,
                float* out, void* hip_stream);

}  // namespace milo
