/*
 * tide.h -- C ABI of the paged-KV resume-attention library for AMD MI355X (gfx950).
 *
 * What the library computes (TideRL, arXiv 2608.10402):
 *   A multi-turn agent task pauses while the environment runs, then resumes with
 *   a longer context.  When the task's KV cache was kept resident (Continuous Task
 *   Batching, Section 4, and its resume-with-cache-locality rule in Section 4.2),
 *   the resume only has to run attention for the newly appended observation/action
 *   tokens against the retained prefix.  When the cache was evicted (challenge C1
 *   in Section 2.2) or invalidated by a weight update ("cache-free task migration",
 *   Section 5.2), the whole history is prefilled again.  Between environment turns
 *   the task decodes its next action one token at a time (Section 2.1).
 *
 *   The four compute entry points below are exactly these steps:
 *     tide_kv_append          write new tokens' K/V into the shared page pool
 *     tide_extend_attn        attention of the new tokens over retained prefix + themselves
 *     tide_decode_attn        one query token per task over its whole context (split-K)
 *     tide_full_prefill_attn  causal attention over the whole sequence (the recompute path)
 *   the same steps with the KV-append fused into the attention:
 *     tide_extend_append_attn tide_kv_append of the new tokens + tide_extend_attn
 *     tide_decode_append_attn tide_kv_append of one token per task + tide_decode_attn
 *   and decode for GRPO groups whose trajectories share a prompt prefix:
 *     tide_decode_attn_shared tide_decode_attn, reading each shared prefix once per group
 *
 *   The attention itself is standard scaled dot-product attention (Vaswani et al.,
 *   2017), which the paper uses but does not restate: for a query row at absolute
 *   position t of task b and query head h,
 *       s_p = sm_scale * <q, k_p>           for key positions p = 0 .. t
 *       o   = sum_p softmax(s)_p * v_p,     lse = log(sum_p exp(s_p))  (natural log)
 *   with k_p, v_p taken from KV head floor(h / G), G = num_q_heads / num_kv_heads
 *   (grouped-query attention).  Causality is bottom-right aligned: the j-th new token
 *   of a task with prefix length P sits at position P + j and sees keys 0 .. P + j.
 *
 * Memory layout (all device buffers are owned by the caller):
 *   element type     bf16 (raw 16-bit brain-float bit patterns) for Q, K, V, O;
 *                    fp32 for LSE.
 *   k_pool, v_pool   bf16 [num_pages][num_kv_heads][page_size][head_dim] each
 *                    (one (page, kv-head) block is page_size token rows of head_dim
 *                    contiguous values; the kernels transpose V operands in LDS)
 *   block_table      int32 [num_tasks][bt_stride], row-major, device memory.  Entry i of
 *                    row b is the physical page holding logical positions
 *                    [i*page_size, (i+1)*page_size) of task b.  Only the first
 *                    ceil(len_b / page_size) entries of a row are read.
 *   token tensors    packed ragged rows: task b owns rows [indptr_b, indptr_{b+1}) where
 *                    indptr is the exclusive prefix sum of the per-task token counts in
 *                    task order.  q/out: bf16 [rows][num_q_heads][head_dim];
 *                    k_new/v_new: bf16 [rows][num_kv_heads][head_dim];
 *                    lse: fp32 [rows][num_q_heads] (may be NULL).
 *   lengths          HOST arrays of int32, read synchronously during the call (the
 *                    scheduler that owns task footprints lives on the host, Section 4.1).
 *   workspace        device scratch owned by the caller, at least tide_workspace_size()
 *                    bytes; it must not be shared by two calls in flight at once.
 *   stream           a hipStream_t passed as void*; NULL means the default stream.
 *
 * Supported shapes: head_dim in {64, 128}; page_size == 16; num_q_heads a multiple of
 * num_kv_heads with G = num_q_heads / num_kv_heads in [1, 16]; num_kv_heads <= 65536.
 * Anything else returns TIDE_ERR_UNSUPPORTED.
 *
 * Semantics guaranteed by every attention entry point:
 *   - Pool slots at or beyond a task's current length, and pages not listed in its
 *     block-table prefix, never influence the result, even if they hold NaN or Inf.
 *   - The result does not depend on which physical pages hold the data (bitwise, for a
 *     fixed split count), and repeated calls on the same inputs are bitwise identical.
 *   - A physical page id outside [0, num_pages) is never dereferenced: the kernels
 *     skip it and set an error flag in the workspace; with the environment variable
 *     TIDE_DEBUG_CHECKS=1 the call synchronizes the stream and returns
 *     TIDE_ERR_PAGE_RANGE when the flag is set.
 *
 * Calls enqueue work on `stream` and return without synchronizing (except under
 * TIDE_DEBUG_CHECKS=1).  Device faults surface at the caller's next synchronization.
 * No C++ exception or abort crosses this interface.  The library never allocates
 * device memory at run time (its one static device array, the scratch of
 * tide_decode_attn_noalloc, comes with the code object); it keeps a small pinned,
 * device-mapped host staging ring (created lazily, released by tide_shutdown) from which
 * a copy kernel on `stream` moves each call's work list into the workspace.  Calls that
 * take a workspace are thread-safe when each call in flight has its own workspace.
 */
#ifndef TIDE_H_
#define TIDE_H_

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define TIDE_API __attribute__((visibility("default")))
#else
#define TIDE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
enum {
  TIDE_OK = 0,
  TIDE_ERR_INVALID_ARG = -1, /* null pointer, non-positive dimension, negative length */
  TIDE_ERR_UNSUPPORTED = -2, /* head_dim / page_size / GQA ratio outside the supported set */
  TIDE_ERR_CAPACITY = -3,    /* ceil(len/page_size) > bt_stride, or workspace too small */
  TIDE_ERR_HIP = -4,         /* a HIP runtime call or kernel launch failed */
  TIDE_ERR_PAGE_RANGE = -5   /* a block-table page id was outside [0, num_pages) (debug mode) */
};

/* Operation selector for tide_workspace_size. */
enum {
  TIDE_OP_KV_APPEND = 1,
  TIDE_OP_EXTEND = 2,
  TIDE_OP_DECODE = 3,
  TIDE_OP_FULL_PREFILL = 4
};

/* Attention shape shared by all calls. */
typedef struct tide_dims {
  int32_t num_q_heads;  /* Hq */
  int32_t num_kv_heads; /* Hkv; Hq % Hkv == 0 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t page_size;    /* tokens per page: 16 */
  float sm_scale;       /* softmax scale, usually 1/sqrt(d); must be finite and > 0 */
} tide_dims;

/*
 * Bytes of device workspace the operation needs for these host lengths.
 *   op == TIDE_OP_KV_APPEND / TIDE_OP_EXTEND: lens_a = prefix_lens, lens_b = extend_lens
 *   op == TIDE_OP_DECODE:                     lens_a = kv_lens,     lens_b ignored
 *   op == TIDE_OP_FULL_PREFILL:               lens_a = seq_lens,    lens_b ignored
 * num_splits is used by TIDE_OP_DECODE only (0 = automatic; see tide_decode_attn).
 * The size depends only on the arguments, never on device state.
 */
TIDE_API int tide_workspace_size(int op, int32_t num_tasks, const int32_t* lens_a, const int32_t* lens_b,
                        const tide_dims* dims, int32_t num_splits, size_t* bytes_out);

/* The launch a call with these arguments makes (diagnostics: which kernel variant runs,
 * and how the work is cut).  Same arguments as tide_workspace_size; fills *out. */
typedef struct tide_plan_info {
  int32_t num_items;        /* work items (workgroups for extend/prefill, waves for decode) */
  int32_t waves_per_group;  /* waves per workgroup of the main kernel */
  int32_t split;            /* extend/prefill: 1 when split-KV chunks and a merge run */
  int32_t max_splits;       /* decode: the most splits of any task */
  int32_t merge_in_kernel;  /* decode: 1 when the split kernel merges (no merge kernel) */
  int32_t reserved;
  size_t workspace_bytes;
} tide_plan_info;
TIDE_API int tide_plan_info_get(int op, int32_t num_tasks, const int32_t* lens_a,
                        const int32_t* lens_b, const tide_dims* dims, int32_t num_splits,
                        tide_plan_info* out);

/*
 * KV-append: store the K/V of each task's new tokens into its pages (the retained
 * state that Continuous Task Batching keeps resident, Section 4).
 * For task b, new token j (0 <= j < extend_lens[b]) sits at position
 * pos = prefix_lens[b] + j and row r = indptr_b + j of k_new/v_new; for every KV head g:
 *     k_pool[BT[b][pos/16]][g][pos%16][:] = k_new[r][g][:]
 *     v_pool[BT[b][pos/16]][g][pos%16][:] = v_new[r][g][:]
 * The copy is bit-exact; no other pool byte is written.  Two tasks must not map the
 * same (page, slot); if they do, the result for that slot is unspecified.
 */
TIDE_API int tide_kv_append(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                   int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                   int32_t num_tasks, const int32_t* prefix_lens, const int32_t* extend_lens,
                   const tide_dims* dims, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Extend attention: resume of tasks whose KV was retained (Section 4.2; the cache hit
 * that avoids the recompute of challenge C1, Section 2.2).  For each task b the
 * extend_lens[b] query rows at positions prefix_lens[b] .. prefix_lens[b]+extend_lens[b]-1
 * attend causally to keys 0 .. their own position, read from the pool only: the new
 * tokens' K/V must already have been appended.  q/out rows are packed by extend_lens.
 * extend_lens[b] == 0 contributes no rows; prefix_lens[b] == 0 is a fresh prefill.
 * A call with too few (task, kv head, token block) work items to keep every compute
 * unit busy is run split-KV: long blocks are cut into key ranges processed in parallel
 * and merged by a second kernel (the workspace then also holds the fp32 partials).  The
 * choice depends only on the lengths and dims, so tide_workspace_size covers it and
 * results stay bitwise repeatable; the environment variable TIDE_EXTEND_SPLIT=0 (never)
 * or =1 (whenever a block spans enough key tiles) overrides it, read on every call.
 */
TIDE_API int tide_extend_attn(const void* q, const void* k_pool, const void* v_pool, int64_t num_pages,
                     const int32_t* block_table, int32_t bt_stride, int32_t num_tasks,
                     const int32_t* prefix_lens, const int32_t* extend_lens,
                     const tide_dims* dims, void* out, float* lse, void* workspace,
                     size_t workspace_bytes, void* stream);

/*
 * Extend attention with the KV-append of the new tokens fused in: the result and the pool
 * contents afterwards are those of tide_kv_append(k_new, v_new, prefix_lens, extend_lens)
 * followed by tide_extend_attn(q, prefix_lens, extend_lens).  Every resume with a retained
 * cache (Section 4.2) appends its new observation/action tokens and then attends over
 * them; fusing removes the append launch and the pool round trip of the new rows.
 *   k_new, v_new  bf16 [rows][Hkv][d], packed by extend_lens like q: the new tokens' K/V.
 * The attention reads keys at or past each task's prefix straight from k_new / v_new, and
 * each (task, kv head, block of new tokens) work item writes its own tokens' rows into
 * their pool slots; no work item of the call reads those slots, so there is no ordering
 * between them.  Workspace: tide_workspace_size(TIDE_OP_EXTEND, ...).  Arguments and errors
 * as tide_extend_attn, plus TIDE_ERR_INVALID_ARG for a NULL k_new / v_new.
 */
TIDE_API int tide_extend_append_attn(const void* q, const void* k_new, const void* v_new,
                            void* k_pool, void* v_pool, int64_t num_pages,
                            const int32_t* block_table, int32_t bt_stride, int32_t num_tasks,
                            const int32_t* prefix_lens, const int32_t* extend_lens,
                            const tide_dims* dims, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Decode attention: one query token per task (the action tokens generated between
 * environment turns, Section 2.1) over its whole context of kv_lens[b] >= 1 positions,
 * which include the token itself (append it first).  q/out: bf16 [num_tasks][Hq][d];
 * lse: fp32 [num_tasks][Hq] or NULL.  The context is split into chunks processed in
 * parallel and merged by log-sum-exp weights (split-K).  num_splits == 0 chooses the
 * chunk size automatically; num_splits > 0 caps the number of chunks per task at that
 * value.  Results for different split counts agree to fp32 rounding.
 * Every K/V page is streamed with the non-temporal cache hint, since each task's context
 * is read once.  Tasks whose block tables share pages (a GRPO group's prompt) should go
 * through tide_decode_attn_shared, which reads a shared prefix once per group; here each
 * task re-reads it from HBM.
 */
TIDE_API int tide_decode_attn(const void* q, const void* k_pool, const void* v_pool, int64_t num_pages,
                     const int32_t* block_table, int32_t bt_stride, int32_t num_tasks,
                     const int32_t* kv_lens, const tide_dims* dims, int32_t num_splits,
                     void* out, float* lse, void* workspace, size_t workspace_bytes,
                     void* stream);

/*
 * Decode step with its KV-append fused in: the result and the pool contents afterwards
 * are those of tide_kv_append(k_new, v_new, prefix_lens = kv_lens - 1, extend_lens = 1)
 * followed by tide_decode_attn(q, kv_lens).  Every generated token of a resumed task is
 * such a one-token resume (Section 2.1); fusing removes the append launch and its
 * round trip through HBM from each step.
 *   k_new, v_new  bf16 [num_tasks][Hkv][d]: K/V of each task's newest token, which sits
 *                 at position kv_lens[b] - 1 (its page must be mapped in the block table;
 *                 its slot is overwritten).
 * The split that covers that position takes the token straight from k_new / v_new and
 * writes it into its slot; no other split reads the slot, so there is no ordering
 * between workgroups.  Workspace: tide_workspace_size(TIDE_OP_DECODE, ...).  Arguments
 * and errors as tide_decode_attn, plus TIDE_ERR_INVALID_ARG for a NULL k_new / v_new.
 * In debug mode an invalid page id of the newest token is reported like any other.
 */
TIDE_API int tide_decode_append_attn(const void* q, const void* k_new, const void* v_new,
                            void* k_pool, void* v_pool, int64_t num_pages,
                            const int32_t* block_table, int32_t bt_stride, int32_t num_tasks,
                            const int32_t* kv_lens, const tide_dims* dims, int32_t num_splits,
                            void* out, float* lse, void* workspace, size_t workspace_bytes,
                            void* stream);

/*
 * Decode attention that allocates nothing, for callers that cannot allocate device or
 * pinned memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, result and errors as tide_decode_attn, without the
 * workspace: the work list and split partials live in a static device array of
 * TIDE_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on until the
 * process ends.  A call whose tide_workspace_size(TIDE_OP_DECODE, ...) exceeds that
 * returns TIDE_ERR_CAPACITY before any device work.  The work list is copied into the
 * array with hipMemcpyAsync from pageable host memory, so the call may wait for work
 * already queued on `stream`.  Every call on one GPU uses the same array: two calls in
 * flight at once on one GPU (on different streams, or from different threads) race and
 * give undefined results; serialize them on one stream.
 */
#define TIDE_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
TIDE_API int tide_decode_attn_noalloc(const void* q, const void* k_pool, const void* v_pool,
                             int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                             int32_t num_tasks, const int32_t* kv_lens, const tide_dims* dims,
                             int32_t num_splits, void* out, float* lse, void* stream);

/*
 * Decode attention for tasks grouped by a shared prompt prefix.  GRPO samples a group of
 * trajectories per task (Section 2.1), and Continuous Task Batching resumes them with
 * group affinity so that they keep sharing the prefix pages (Section 4.2).  The result
 * is that of tide_decode_attn on the same arguments; only the pages of a shared prefix
 * are read once per group of up to 16 / G trajectories instead of once per trajectory.
 *   group_start  host int32 [num_groups + 1]: group g is tasks group_start[g] ..
 *                group_start[g+1] - 1 (consecutive, non-empty; group_start[0] == 0,
 *                group_start[num_groups] == num_tasks; a lone task is a group of one)
 *   shared_lens  host int32 [num_groups]: the first shared_lens[g] positions of every
 *                member are the same physical pages (equal leading block-table entries)
 *                holding the same K/V; a multiple of the page size, at most kv_len - 1 of
 *                every member (the decoded token is each trajectory's own); 0 = nothing
 *                shared.  The shared pages are read through the group's first task.
 * num_splits as in tide_decode_attn (the shared prefix and a task's own keys are split
 * separately, so a task may get one split more).  Workspace: tide_workspace_size_shared.
 * Errors: TIDE_ERR_INVALID_ARG for a malformed group table or shared length.
 */
TIDE_API int tide_decode_attn_shared(const void* q, const void* k_pool, const void* v_pool,
                            int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                            int32_t num_tasks, const int32_t* kv_lens, int32_t num_groups,
                            const int32_t* group_start, const int32_t* shared_lens,
                            const tide_dims* dims, int32_t num_splits, void* out, float* lse,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace tide_decode_attn_shared needs for these host arguments. */
TIDE_API int tide_workspace_size_shared(int32_t num_tasks, const int32_t* kv_lens,
                               int32_t num_groups, const int32_t* group_start,
                               const int32_t* shared_lens, const tide_dims* dims,
                               int32_t num_splits, size_t* bytes_out);

/*
 * Full re-prefill attention: causal attention over all seq_lens[b] positions of each
 * task, the recomputation an evicted or invalidated cache forces (challenge C1,
 * Section 2.2; fresh prefill after a weight sync, Section 5.2).  Identical to
 * tide_extend_attn with prefix_lens = 0 and extend_lens = seq_lens.
 */
TIDE_API int tide_full_prefill_attn(const void* q, const void* k_pool, const void* v_pool,
                           int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                           int32_t num_tasks, const int32_t* seq_lens, const tide_dims* dims,
                           void* out, float* lse, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Human-readable text for a status code (static storage, never NULL). */
TIDE_API const char* tide_status_string(int status);

/* Release the pinned host staging ring.  Safe to call at any time when no call is in
 * flight on another thread; later calls recreate it. */
TIDE_API void tide_shutdown(void);

#ifdef __cplusplus
}
#endif

#endif /* TIDE_H_ */
