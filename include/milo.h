/*
 * milo.h - decode attention over a block-wise low-rank KV cache (C ABI).
 *
 * The operation (MILO, Sec. 4.2 Eq. 3, Sec. 4.4 Alg. 1 inference stage, Sec. 4.1
 * Eq. 1): a many-shot context is split into blocks; block b of T_b tokens keeps
 * its keys and values as factors
 *        K_b ~ P^K_b R^K_b,      V_b ~ P^V_b R^V_b,
 * where P is T_b x r and R is r x (H_kv*d), with the diagonal of singular values
 * already multiplied into P (or split between P and R in any way).  Ranks may
 * differ per block and between K and V (Sec. 4.3, Sec. 4.4).  The columns of R
 * are head-major: KV head g owns columns g*d .. g*d+d-1.  A decode step attends
 * every query token to the selected blocks (the retriever's output, Alg. 1) and
 * to that request's own uncompressed KV (the "dense tail"):
 *        o_{i,h} = softmax(scale * [K_sel; K_tail,i] q_{i,h}) [V_sel; V_tail,i]
 * with query head h reading KV head g = h / (H_q / H_kv).  The library computes
 * this in each block's rank space (project the query through R^K, score against
 * P^K rows, accumulate weights times P^V rows, up-project through R^V) and merges
 * blocks and tail with a log-sum-exp reduction; it never rebuilds K or V.
 *
 * Conventions
 *  - bf16 values are passed as uint16_t bit patterns; all buffers row-major and
 *    C-contiguous.  Output is fp32.  Accumulation is fp32.
 *  - "host" pointers are ordinary CPU memory; "device" pointers are HIP device
 *    memory of the current device (e.g. torch tensors on cuda:N).
 *  - Every function returns a status code (MILO_OK = 0, negative on error) and
 *    never throws.  On error, milo_last_error() holds a message for the calling
 *    thread.  Argument checks happen on the host before any GPU work is queued.
 *  - milo_attend_decode is asynchronous: it only enqueues kernels on hip_stream
 *    (NULL = the default stream).  Errors inside kernels surface at the next
 *    synchronisation.
 */
#ifndef MILO_H
#define MILO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MILO_OK 0
#define MILO_ERR_INVALID_ARG (-1)   /* bad pointer, shape, rank, id or length   */
#define MILO_ERR_OUT_OF_MEMORY (-2) /* device allocation failed or over the cap */
#define MILO_ERR_HIP (-3)           /* a HIP runtime call failed                */
#define MILO_ERR_UNSUPPORTED (-4)   /* valid input this library does not handle */

/* Opaque cache handle: owns one device buffer with every block's factors in the
 * library's packed layout, plus per-call workspace. */
typedef struct milo_cache milo_cache;

/* Shape of a low-rank cache (Sec. 4.2: per-block factors, Sec. 4.3: per-block
 * ranks).  All arrays are host memory, read during milo_cache_create only.
 *   n_blocks      number of blocks N >= 1
 *   n_kv_heads    H_kv >= 1
 *   head_dim      d, 64 or 128 (others return MILO_ERR_UNSUPPORTED)
 *   block_tokens  [n_blocks] T_b >= 1
 *   rank_k/v      [n_blocks] 1 <= r <= min(T_b, H_kv*d), at most 1024 (larger
 *                 ranks return MILO_ERR_UNSUPPORTED).  The latent route handles
 *                 r <= 896; a selected block of higher rank (full rank at
 *                 H_kv*d = 1024) is always attended by reconstruction
 *                 (milo_cache_set_path), so INT8 caches stay at r <= 896 and
 *                 milo_attend_decode_noalloc refuses such blocks. */
typedef struct milo_cache_desc {
  int32_t n_blocks;
  int32_t n_kv_heads;
  int32_t head_dim;
  const int32_t* block_tokens;
  const int32_t* rank_k;
  const int32_t* rank_v;
  int32_t p_format;  /* MILO_P_BF16 (0) or MILO_P_INT8 (1), see below */
} milo_cache_desc;

/* Storage of the P factors (p_format).  MILO_P_INT8 combines the low-rank cache
 * with INT8 quantisation (Sec. 5.3, Table 2): P^K and P^V are stored as int8
 * codes with one fp32 scale per token row, s_t = max_k |P[t][k]| / 127 and
 * c[t][k] = round-to-nearest-even(P[t][k] / s_t) (fp32, correctly rounded
 * division), so P[t][k] is replaced by s_t c[t][k]; the R factors stay bf16.
 * This halves the bytes of P (1 byte per element plus 8 bytes per token).
 * Attention then computes exactly with the dequantised factors s_t c[t][k]
 * (codes exact in bf16, scales applied in fp32).  Creation refuses a P factor
 * with a non-finite value (INVALID_ARG). */
#define MILO_P_BF16 0
#define MILO_P_INT8 1

/* Build a cache from per-block factors (LC.Store of Alg. 1, encoding stage, with
 * the singular values folded into P).
 *   pk, pv        [n_blocks] pointers to bf16 P^K_b [T_b][rank_k_b], P^V_b [T_b][rank_v_b]
 *   rk, rv        [n_blocks] pointers to bf16 R^K_b [rank_k_b][H_kv*d], R^V_b [rank_v_b][H_kv*d]
 *   src_on_device 0: the factor pointers are host memory; 1: device memory.
 *                 The pointer arrays themselves are always host memory.
 *   hip_stream    stream used for the copies and packing kernels.
 *   out           receives the handle (set to NULL on failure).
 * Synchronous: when it returns the caller may free or reuse its factor buffers.
 * Errors: INVALID_ARG (null pointer, bad shape or rank), UNSUPPORTED (head_dim,
 * rank above the supported maximum), OUT_OF_MEMORY (hipMalloc failed, or the
 * total exceeds the byte cap in the MILO_MAX_DEVICE_BYTES environment variable),
 * HIP_ERROR. */
int milo_cache_create(const milo_cache_desc* desc, const uint16_t* const* pk,
                      const uint16_t* const* rk, const uint16_t* const* pv,
                      const uint16_t* const* rv, int src_on_device, void* hip_stream,
                      milo_cache** out);

/* One decode step of attention over the selected blocks plus each request's
 * dense tail (Alg. 1 inference stage; Eq. 1).  The step's work plan gives every
 * workgroup a program that must fit in LDS; when the programs would not fit
 * (or exceed the byte cap in the MILO_MAX_PROGRAM_BYTES environment variable,
 * read when a plan is built) the work is split over several launches.
 *   cache         from milo_cache_create, on the current device.
 *   block_table   host [n_sel] distinct block ids in [0, n_blocks) (the retriever's
 *                 selection; any order gives the same result up to rounding).
 *                 May be NULL when n_sel == 0 (tail-only attention).
 *   n_q           decode batch: independent query tokens sharing the context, >= 1.
 *   n_q_heads     H_q, a multiple of H_kv with H_q / H_kv <= 16.
 *   q             device bf16 [n_q][H_q][d].
 *   tail_k/v      device bf16 [n_q][tail_cap][H_kv][d]; request i uses its first
 *                 tail_len[i] rows.  May be NULL when tail_cap == 0.
 *   tail_len      host [n_q], 0 <= tail_len[i] <= tail_cap; may be NULL when
 *                 tail_cap == 0.  Every request must see at least one key
 *                 (n_sel > 0 or tail_len[i] > 0).
 *   scale         softmax temperature, usually 1/sqrt(d) (Eq. 1); finite.
 *   out           device fp32 [n_q][H_q][d], fully overwritten.
 *   hip_stream    stream the work is queued on.
 * q, tail_k, tail_v and out are borrowed until the queued work completes.  The
 * cache's workspace is shared by its calls: calls on one cache must be ordered on
 * one stream (calls on different streams race).
 * Work plan: built on the host when the block table, n_q, H_q or the planned
 * tail capacity changes, where the capacity is the longest tail rounded up to a
 * power of two of 256-token chunks, at most tail_cap.  A decode loop whose tails
 * grow by a token per call therefore reuses its plan until the longest tail
 * doubles: the tail lengths themselves travel in the kernel arguments (for
 * n_q <= 256; larger batches copy them to the device in stream order).  A
 * rebuild uploads in stream order without waiting for the device, unless the
 * plan outgrows its buffer; workspace growth also waits for the stream.
 * Errors: INVALID_ARG, UNSUPPORTED, OUT_OF_MEMORY, HIP_ERROR. */
int milo_attend_decode(milo_cache* cache, const int32_t* block_table, int32_t n_sel,
                       int32_t n_q, int32_t n_q_heads, const uint16_t* q,
                       const uint16_t* tail_k, const uint16_t* tail_v,
                       const int32_t* tail_len, int32_t tail_cap, float scale, float* out,
                       void* hip_stream);

/* milo_attend_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, kernels and results, but the call's workspace (work plan,
 * partial results, tail lengths of batches above 256 requests) lives in a fixed
 * 64 MiB scratch array of the library, one copy per GPU, held until the process
 * ends; the call makes no device allocation and no hipFree (the plan is built in
 * host memory and copied in stream order).  Limits: an 8 MiB plan, 55 MiB of
 * partial results (n_q * H_q columns x slots x (4 d + 8) bytes; e.g. the
 * 7B- and 32B-shaped layers fit, a 14B-shaped 64-query layer does not) and
 * 262144 requests; larger calls return MILO_ERR_UNSUPPORTED before queuing
 * anything.  Every call on a GPU shares that GPU's scratch and it keeps the
 * last call's contents (nothing in it needs clearing): calls that overlap on one
 * GPU race, so order them on one stream.  Kernel timing (milo_timing_*) does not
 * record these calls.  Errors: as milo_attend_decode. */
int milo_attend_decode_noalloc(milo_cache* cache, const int32_t* block_table, int32_t n_sel,
                               int32_t n_q, int32_t n_q_heads, const uint16_t* q,
                               const uint16_t* tail_k, const uint16_t* tail_v,
                               const int32_t* tail_len, int32_t tail_cap, float scale,
                               float* out, void* hip_stream);

/* Prefill of one request: a chunk of n_tok consecutive query tokens attends to
 * the selected blocks plus the request's dense tail, causally among its own
 * tokens (Alg. 1 inference stage with a multi-token input query Q; Eq. 1).
 * Token j (0-based) sees the blocks and tail rows [0, tail_base + j + 1): the
 * tail_base rows that precede the chunk and the chunk's own first j + 1 tokens,
 * whose keys and values the caller has stored at rows tail_base ..
 * tail_base + n_tok - 1.
 *   n_tok         tokens in the chunk, >= 1.
 *   q             device bf16 [n_tok][H_q][d].
 *   tail_k/v      device bf16 [tail_cap][H_kv][d], one tail read by every token.
 *   tail_base     rows of the tail before the chunk, >= 0; tail_base + n_tok <= tail_cap.
 *   out           device fp32 [n_tok][H_q][d], fully overwritten.
 * cache, block_table, n_sel, n_q_heads, scale, hip_stream, ownership and errors
 * as for milo_attend_decode (the work is that of a decode step whose n_tok
 * requests share one tail with lengths tail_base + 1 .. tail_base + n_tok). */
int milo_attend_prefill(milo_cache* cache, const int32_t* block_table, int32_t n_sel,
                        int32_t n_tok, int32_t n_q_heads, const uint16_t* q,
                        const uint16_t* tail_k, const uint16_t* tail_v,
                        int32_t tail_base, int32_t tail_cap, float scale, float* out,
                        void* hip_stream);

/* How a cache's blocks are attended (Sec. 4.5 inference path).
 *   MILO_PATH_LATENT       (default) every block in its rank space (Eq. 1 with
 *                          q.k = (R^K q).p): the query is projected through R^K,
 *                          scored against P^K, the weights pass through P^V and
 *                          the result is lifted through R^V.
 *   MILO_PATH_RECONSTRUCT  every selected block is first rebuilt at full rank,
 *                          K_b = P^K_b R^K_b and V_b = P^V_b R^V_b (Alg. 1
 *                          full-rank reconstruction; fp32 accumulation, keys
 *                          stored as fp16 (saturated at +-65504), values as
 *                          bf16), into a per-call buffer of the cache
 *                          (4 T_pad H_kv d bytes per selected block, kept and
 *                          grown like the rest of the workspace), and then
 *                          attended as uncompressed keys and values.
 *   MILO_PATH_AUTO         per block and call, whichever an MI355X cost model
 *                          (fitted to measured kernel times) expects to be
 *                          clearly faster: reconstruction pays for blocks of
 *                          high rank attended by many query columns (the
 *                          latent route costs ~ r N (T + d), reconstruction
 *                          ~ r T H_kv d + T H_kv d + N T d; N = n_q H_q), e.g.
 *                          the ranks above ~400 of a 14B-shaped 64-query step.
 * Both routes compute the same attention up to rounding.  A plan with any
 * reconstructed block cuts the query columns per KV head.  INT8 caches attend
 * latent only (UNSUPPORTED for the other paths), and so does
 * milo_attend_decode_noalloc (AUTO attends latent there; RECONSTRUCT returns
 * UNSUPPORTED).  The setting applies from the next call on; calls queued
 * earlier are not affected.  Errors: INVALID_ARG (NULL cache, unknown path),
 * UNSUPPORTED.
 * milo_cache_recon_blocks: how many blocks the plan of the cache's last
 * milo_attend_decode / milo_attend_prefill call reconstructs. */
#define MILO_PATH_LATENT 0
#define MILO_PATH_RECONSTRUCT 1
#define MILO_PATH_AUTO 2
int milo_cache_set_path(milo_cache* cache, int32_t path);
int milo_cache_recon_blocks(const milo_cache* cache, int32_t* n);

/* Pre-RoPE keys.  The paper factorises keys before the rotary position
 * embedding is applied (Sec. 3 studies the low rank of pre-RoPE keys); such a
 * cache cannot be attended in rank space (the rotation does not commute with
 * R^K), so after this call every selected block is reconstructed (Sec. 4.5,
 * Alg. 1 full-rank reconstruction) and its keys are rotated before attention,
 * whatever milo_cache_set_path says: token t of block b sits at position
 * block_pos[b] + t and its key, per KV head, becomes
 *        (u, v) -> (u cos a - v sin a,  v cos a + u sin a),  a = p theta^(-2j/d)
 * for each pair u = k[j], v = k[j + d/2], j < d/2 (the rotate-half arrangement
 * of the Qwen2 models the paper evaluates).  The rotation is applied to the
 * fp32 reconstruction, before its rounding to fp16: the angle is formed in turns,
 * p theta^(-2j/d) / (2 pi), in fp64, reduced to [0, 1) and its sine and
 * cosine taken in fp32 by the hardware's turn-based instructions (error below
 * ~1e-6 at any int32 position).
 * The queries and the dense tail's keys are taken as already rotated (at the
 * query's own position), as a serving stack stores them.
 *   theta      rotary base (Qwen2.5: 1e6), finite and > 1; 0 turns the
 *              rotation off again (keys attended as stored).
 *   block_pos  host [n_blocks] first-token positions, 0 <= block_pos[b] and
 *              block_pos[b] + T_b rounded up to 256 <= 2^31 - 1; NULL places
 *              the blocks one after another in id order from position 0.
 *              Blocks may overlap or leave gaps (a retriever's reordering).
 * Uploads d/2 frequencies (fp64) and waits for the device before freeing the
 * previous ones; later calls rebuild their plan.  INT8 caches (attended latent
 * only) return UNSUPPORTED, and so does milo_attend_decode_noalloc on such a
 * cache when a block is selected.
 * Errors: INVALID_ARG (NULL cache, theta, positions), UNSUPPORTED,
 * OUT_OF_MEMORY, HIP_ERROR. */
int milo_cache_set_rope(milo_cache* cache, double theta, const int64_t* block_pos);

/* Entropy-based rank allocation of the encoder (Sec. 4.3): the per-block ranks
 * r_b that maximise the retained spectral information sum_b H_b(r_b), with
 * H_b(r) = sum_{j<=r} log(1 + sigma_{b,j}^2 / eps^2) (Eq. 5), subject to
 * sum_b r_b <= r_total and r_min <= r_b <= r_max (Eq. 6), as the greedy over
 * marginal gains of Eq. 7 assigns them: every block starts at its floor and
 * each further unit goes to the block with the largest next singular value.
 * The result does not depend on eps (the gain is increasing in sigma), so eps
 * is not an argument.  A block cannot exceed its own number of singular values:
 * its floor is min(r_min, n_sv[b]) and its cap min(r_max, n_sv[b]); when every
 * block reaches its cap the sum stays below r_total; equal singular values go
 * to the lower block index first.  Run it once for the key spectra and once for
 * the value spectra (Eq. 4 counts both) to get rank_k and rank_v for
 * milo_cache_create.
 *   sigma      device fp32 [n_blocks][ld]; row b holds block b's singular values
 *              in its first n_sv[b] columns, finite, >= 0 and non-increasing
 *              (the rest of the row is not read).
 *   ld         row stride in elements, >= 1 and >= every n_sv[b].
 *   n_blocks   >= 1.
 *   n_sv       host [n_blocks], 0 <= n_sv[b] <= ld (min(T_b, H_kv*d) for an SVD).
 *   r_total    rank budget R_tot, at least sum_b min(r_min, n_sv[b]).
 *   r_min/max  0 <= r_min <= r_max.
 *   ranks      host [n_blocks] out.
 *   hip_stream stream the kernels run on; the call waits for them (synchronous).
 * Allocates and frees a small device workspace per call.  Errors: INVALID_ARG
 * (NULL pointer, bad bounds, budget below the floors, or a row that is not
 * finite, non-negative and non-increasing: the message names the lowest such
 * block; ranks is then untouched), UNSUPPORTED (2^31 or more candidate values),
 * OUT_OF_MEMORY, HIP_ERROR. */
int milo_allocate_ranks(const float* sigma, int64_t ld, int32_t n_blocks, const int32_t* n_sv,
                        int64_t r_total, int32_t r_min, int32_t r_max, int32_t* ranks,
                        void* hip_stream);

/* Encoder, per-block truncated SVD (Sec. 4.2 Eq. 3, Alg. 1 encoding stage).
 * milo_block_svd: for every block's keys (or values) K_b, the singular values and
 * right singular vectors, K_b = U diag(sigma) V^T: the Gram matrix K_b^T K_b in
 * fp32, its eigenvectors by block Jacobi (blocks of 32 indices; rotations until
 * every off-diagonal entry is below 1e-6 of its diagonal geometric mean or
 * 1e-10 of the trace, at most 30 sweeps), the eigenvalues sorted in descending
 * order,
 * sigma = sqrt(max(lambda, 0)).  The Gram matrix squares the condition number:
 * in fp32 the eigenvalues carry an absolute error of about 1e-7 .. 1e-6
 * lambda_max, so singular values far below 1e-3 sigma_max are correspondingly
 * coarse.
 *   k        host [n_blocks] pointers to device bf16 K_b [T_b][d_model] (row-major)
 *   n_blocks 1 .. 65535
 *   tokens   host [n_blocks] T_b >= 1
 *   d_model  D = H_kv * d, 1 <= D <= 1024 (larger: UNSUPPORTED)
 *   sigma    device fp32 [n_blocks][D], out: non-increasing (values past
 *            min(T_b, D) are ~0); feed to milo_allocate_ranks (n_sv = min(T_b, D))
 *   vt       device fp32 [n_blocks][D][D], out: row j = right singular vector of sigma_j
 * Synchronous (allocates and frees a workspace of at most ~2 GiB: blocks are
 * processed in groups that fit it, at least one at a time).
 * milo_block_factors: the truncated factors of rank r_b with the singular values
 * folded into P (Eq. 3 with Sigma in the left factor): P_b = K_b V_r = U_r Sigma_r
 * and R_b = V_r^T, in bf16 (fp32 accumulation), the inputs of milo_cache_create.
 *   vt       from milo_block_svd; ranks host [n_blocks], 1 <= r_b <= min(T_b, D)
 *   p_out    host [n_blocks] pointers to device bf16 [T_b][r_b], out
 *   r_out    host [n_blocks] pointers to device bf16 [r_b][D], out
 * Synchronous.  Errors (both): INVALID_ARG (NULL pointer, bad count or rank),
 * UNSUPPORTED (d_model), OUT_OF_MEMORY, HIP_ERROR.
 * milo_block_svd_sweeps: the largest number of Jacobi sweeps a block of the
 * last milo_block_svd call needed (30 means some block stopped at the cap).
 * milo_block_svd_flops: the fp32 flops that call executed in its Gram products
 * (2 T_b D^2 per block) and in the 64 x 64 x 64 products of its block rotations
 * (counted on the device as they run); the scalar rotations inside the 64 x 64
 * subproblems are not counted.  Both: INVALID_ARG for NULL. */
int milo_block_svd(const uint16_t* const* k, const int32_t* tokens, int32_t n_blocks, int32_t d_model,
                   float* sigma, float* vt, void* hip_stream);
int milo_block_factors(const uint16_t* const* k, const int32_t* tokens, int32_t n_blocks,
                       int32_t d_model, const float* vt, const int32_t* ranks,
                       uint16_t* const* p_out, uint16_t* const* r_out, void* hip_stream);
int milo_block_svd_sweeps(int32_t* sweeps);
int milo_block_svd_flops(double* flops);

/* Release the cache and its device memory (synchronises the device first).
 * NULL is accepted and ignored. */
void milo_cache_free(milo_cache* cache);

/* Message describing the last error on the calling thread ("" if none). The
 * pointer stays valid until the thread's next library call. */
const char* milo_last_error(void);

/* Bytes of device memory the cache holds for its packed factors. Returns
 * INVALID_ARG for NULL arguments. */
int milo_cache_device_bytes(const milo_cache* cache, int64_t* bytes);

/* INT8 P factors: copy block `block`'s stored codes and scales of P^K (which = 0)
 * or P^V (which = 2) to host memory: codes [T_b][rank] row-major, scales [T_b].
 * Synchronous.  Errors: INVALID_ARG (NULL argument, a cache with bf16 P factors,
 * bad block or which), HIP_ERROR. */
int milo_cache_read_int8(const milo_cache* cache, int32_t block, int32_t which, int8_t* codes,
                         float* scales);

/* Number of work plans milo_attend_decode / milo_attend_prefill have built for
 * this cache so far (a plan is rebuilt when the block table, the batch shape or
 * the planned tail-chunk capacity changes; see milo_attend_decode).  Returns
 * INVALID_ARG for NULL arguments. */
int milo_cache_plan_builds(const milo_cache* cache, int64_t* builds);

/* Copy one stored factor of one block back to host memory in the caller's
 * row-major layout (for checking the packed layout).  which: 0 = P^K, 1 = R^K,
 * 2 = P^V, 3 = R^V.  dst: host buffer of the factor's size in uint16_t.
 * Synchronous.  Errors: INVALID_ARG (also for P factors stored as INT8),
 * HIP_ERROR. */
int milo_cache_read_factor(const milo_cache* cache, int32_t block, int32_t which,
                           uint16_t* dst);

/* Kernel timing for measurement.  While enabled, every milo_attend_decode
 * has its attention kernel (the fused projection / score / latent-V /
 * up-projection / tail kernel) and its merge kernel record HIP events at their
 * own start and end (the launches record them, so launch gaps are not counted).
 * milo_timing_read synchronises on those events, returns the
 * summed durations in milliseconds and the number of calls, and clears them.
 * Any argument of milo_timing_read may be NULL. */
int milo_timing_enable(int enable);
int milo_timing_read(double* attend_kernel_ms, double* merge_kernel_ms, int64_t* n_calls);
/* The same for the reconstruction kernel of calls that reconstruct blocks:
 * summed milliseconds and the number of such calls since the last read (then
 * cleared); independent of milo_timing_read. */
int milo_timing_read_recon(double* recon_kernel_ms, int64_t* n_calls);
/* The same for milo_allocate_ranks calls made while timing is enabled: summed
 * milliseconds of the whole kernel chain and of its histogram passes, and the
 * number of calls, since the last read (then cleared). */
int milo_timing_read_alloc(double* chain_ms, double* hist_ms, int64_t* n_calls);

#ifdef __cplusplus
}
#endif

#endif /* MILO_H */
