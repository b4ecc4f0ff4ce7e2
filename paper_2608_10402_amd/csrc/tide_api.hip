// The extern "C" entry points declared in include/tide.h: validation and planning on the
// host (plan.cpp), a copy kernel that moves the work lists from a pinned staging ring
// into the caller's workspace, then the kernel launches, all on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdlib.h>
#include <string.h>

#include <sched.h>

#include <algorithm>
#include <chrono>
#include <mutex>
#include <new>
#include <vector>

#include "kernels.h"
#include "plan.h"
#include "tide.h"

namespace tide {
namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kStagingSlots = 16;
// Slots start large and grow by powers of two, so that steady-state calls never
// reallocate: freeing and allocating pinned memory is slow and can stall the device.
constexpr size_t kStagingMin = 2u << 20;

// Pinned, device-mapped host buffers the work lists are staged in.  A kernel on the
// caller's stream copies a slot into the workspace (no DMA-engine copy, so no hand-off
// between engines on every call).  A slot is reused only once that copy has read it:
// each of the copy's workgroups, after all its reads have returned, writes the slot's
// use count into its own flag in coherent host memory, and the host checks the flags
// before it overwrites the slot.  (A completion event recorded behind each copy did the
// same, but delayed the call's next kernel by several microseconds.)
struct StagingSlot {
  void* host = nullptr;
  const void* dev = nullptr;  // the same memory as seen from the device
  size_t cap = 0;
  uint32_t* flags = nullptr;  // one per copy workgroup, coherent host memory
  uint32_t* flags_dev = nullptr;
  uint32_t seq = 0;           // uses of the slot so far
  uint32_t nblocks = 0;       // workgroups of the last copy
  bool pending = false;
};

constexpr int kCopyBytesPerBlock = 256 * 16;

// 16 bytes per thread from the staging slot (host memory) into the workspace; then the
// workgroup's flag.  Every thread's load has returned once it has issued its store (the
// store needs the data), so after the barrier the workgroup has read all it will read.
__global__ __launch_bounds__(256) void stage_copy_kernel(u32x4_t* dst, const u32x4_t* src,
                                                         size_t n16, uint32_t* done, uint32_t seq) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) dst[i] = src[i];
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_store(done + blockIdx.x, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Waits until every workgroup of the slot's last copy has set its flag.  Normally the
// copy finished long ago; if not, this waits like a synchronisation on it would, and
// after a few seconds (TIDE_STAGING_WAIT_US microseconds, if set; tests set 0 to take
// this path) falls back to a device synchronisation (which reports a failed device)
// before giving up.
int wait_slot(StagingSlot& s) {
  auto done = [&] {
    for (uint32_t b = 0; b < s.nblocks; ++b)
      if (__atomic_load_n(s.flags + b, __ATOMIC_ACQUIRE) != s.seq) return false;
    return true;
  };
  if (done()) {
    s.pending = false;
    return TIDE_OK;
  }
  const char* env = getenv("TIDE_STAGING_WAIT_US");
  const long long limit_us = env ? atoll(env) : 5000000LL;
  const auto t0 = std::chrono::steady_clock::now();
  while (!done()) {
    if (std::chrono::steady_clock::now() - t0 >= std::chrono::microseconds(limit_us)) {
      if (hipDeviceSynchronize() != hipSuccess || !done()) return TIDE_ERR_HIP;
      break;
    }
    sched_yield();
  }
  s.pending = false;
  return TIDE_OK;
}

struct DeviceStaging {
  StagingSlot slots[kStagingSlots];
  int next = 0;
};

std::mutex g_mutex;
std::vector<DeviceStaging*> g_staging;  // indexed by device ordinal

// Device scratch of tide_decode_attn_noalloc: the work list and split partials of one
// call, for callers that cannot allocate.  In host code `scratch` names a host-side
// stand-in, never the device array: the device address is taken once per device with
// hipGetSymbolAddress (with that device current) and only that address is used.
static __device__ __align__(256) uint8_t scratch[TIDE_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mutex;
std::vector<void*> g_scratch_ptr;  // device address of `scratch`, indexed by device ordinal

int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TIDE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TIDE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TIDE_OK;
}

bool debug_checks() {
  const char* e = getenv("TIDE_DEBUG_CHECKS");
  return e && e[0] == '1';
}

int upload(const Plan& plan, void* workspace, hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TIDE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mutex);
  if ((int)g_staging.size() <= dev) g_staging.resize(dev + 1, nullptr);
  if (!g_staging[dev]) g_staging[dev] = new DeviceStaging();
  DeviceStaging& ds = *g_staging[dev];
  StagingSlot& s = ds.slots[ds.next];
  ds.next = (ds.next + 1) % kStagingSlots;
  if (s.pending) {
    const int rc = wait_slot(s);
    if (rc != TIDE_OK) return rc;
  }
  const size_t need = plan.blob.size();  // a multiple of kWsAlign
  if (s.cap < need) {
    if (s.host) (void)hipHostFree(s.host);
    if (s.flags) (void)hipHostFree(s.flags);
    s = StagingSlot();
    size_t cap = kStagingMin;
    while (cap < need) cap *= 2;
    const size_t nflags = cap / kCopyBytesPerBlock + 1;
    void* dev_ptr = nullptr;
    void* flags_dev = nullptr;
    if (hipHostMalloc(&s.host, cap, hipHostMallocMapped) != hipSuccess ||
        hipHostGetDevicePointer(&dev_ptr, s.host, 0) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void**>(&s.flags), nflags * sizeof(uint32_t),
                      hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
        hipHostGetDevicePointer(&flags_dev, s.flags, 0) != hipSuccess) {
      if (s.host) (void)hipHostFree(s.host);
      if (s.flags) (void)hipHostFree(s.flags);
      s = StagingSlot();
      return TIDE_ERR_HIP;
    }
    memset(s.flags, 0, nflags * sizeof(uint32_t));
    s.dev = dev_ptr;
    s.flags_dev = static_cast<uint32_t*>(flags_dev);
    s.cap = cap;
  }
  memcpy(s.host, plan.blob.data(), need);
  const size_t n16 = need / 16;
  const uint32_t nblocks = (uint32_t)((n16 + 255) / 256);
  s.seq = s.seq + 1 == 0 ? 1 : s.seq + 1;  // never 0, the flags' initial value
  hipLaunchKernelGGL(stage_copy_kernel, dim3(nblocks), dim3(256), 0, stream,
                     static_cast<u32x4_t*>(workspace), static_cast<const u32x4_t*>(s.dev), n16,
                     s.flags_dev, s.seq);
  if (hipGetLastError() != hipSuccess) return TIDE_ERR_HIP;
  s.nblocks = nblocks;
  s.pending = true;
  return TIDE_OK;
}

int finish(hipError_t launch_status, void* workspace, hipStream_t stream) {
  if (launch_status != hipSuccess) return TIDE_ERR_HIP;
  if (!debug_checks()) return TIDE_OK;
  if (hipStreamSynchronize(stream) != hipSuccess) return TIDE_ERR_HIP;
  int32_t flags = 0;
  if (hipMemcpy(&flags, workspace, sizeof(flags), hipMemcpyDeviceToHost) != hipSuccess)
    return TIDE_ERR_HIP;
  return (flags & 1) ? TIDE_ERR_PAGE_RANGE : TIDE_OK;
}

template <class T>
const T* at(void* ws, size_t off) {
  return reinterpret_cast<const T*>(static_cast<uint8_t*>(ws) + off);
}

template <class T>
T* at_mut(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<uint8_t*>(ws) + off);
}

// Shared path of tide_extend_attn and tide_full_prefill_attn.
// With k_new / v_new (tide_extend_append_attn) the new tokens' K/V are appended by the
// attention kernel itself.
int run_extend(int op, const void* q, const void* k_pool, const void* v_pool, int64_t num_pages,
               const int32_t* block_table, int32_t bt_stride, int32_t num_tasks,
               const int32_t* lens_a, const int32_t* lens_b, const tide_dims* dims, void* out,
               float* lse, void* workspace, size_t workspace_bytes, void* stream,
               const void* k_new = nullptr, const void* v_new = nullptr, bool fused = false) {
  int rc = check_dims(dims);
  if (rc != TIDE_OK) return rc;
  if (num_tasks < 0) return TIDE_ERR_INVALID_ARG;
  if (num_tasks == 0) return TIDE_OK;
  if (num_pages <= 0 || bt_stride <= 0) return TIDE_ERR_INVALID_ARG;
  Plan plan;
  rc = make_plan(op, num_tasks, lens_a, lens_b, *dims, 0, bt_stride, true, &plan);
  if (rc != TIDE_OK) return rc;
  if (plan.num_items == 0) return TIDE_OK;
  if (!q || !k_pool || !v_pool || !block_table || !out || !workspace) return TIDE_ERR_INVALID_ARG;
  if (fused && (!k_new || !v_new)) return TIDE_ERR_INVALID_ARG;
  if (workspace_bytes < plan.total_bytes) return TIDE_ERR_CAPACITY;
  hipStream_t s = static_cast<hipStream_t>(stream);
  rc = upload(plan, workspace, s);
  if (rc != TIDE_OK) return rc;
  ExtendArgs a;
  a.k_new = fused ? static_cast<const uint16_t*>(k_new) : nullptr;
  a.v_new = fused ? static_cast<const uint16_t*>(v_new) : nullptr;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = block_table;
  a.num_pages = num_pages;
  a.bt_stride = bt_stride;
  a.num_q_heads = dims->num_q_heads;
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.scale_log2 = dims->sm_scale * 1.44269504088896340736f;
  a.num_items = plan.num_items;
  a.tasks = at<TaskDesc>(workspace, plan.tasks_off);
  a.items = plan.split ? nullptr : at<ExtendItem>(workspace, plan.items_off);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.error_flags = at_mut<int32_t>(workspace, 0);
  a.chunk_items = plan.split ? at<ExtendChunkItem>(workspace, plan.items_off) : nullptr;
  a.merge_rows = plan.split ? at<MergeRow>(workspace, plan.merge_rows_off) : nullptr;
  a.part_o = plan.split ? at_mut<float>(workspace, plan.part_o_off) : nullptr;
  a.part_ml = plan.split ? at_mut<float>(workspace, plan.part_ml_off) : nullptr;
  a.total_rows = plan.total_rows;
  return finish(launch_extend(a, dims->head_dim, plan.waves, s), workspace, s);
}

// Shared path of tide_decode_attn, tide_decode_append_attn (fused: k_new / v_new) and
// tide_decode_attn_noalloc (in_scratch: the call runs in the static device scratch, its
// work list is copied there with hipMemcpyAsync from the plan's host buffer, and nothing
// is allocated).
int run_decode(const void* q, const void* k_new, const void* v_new, const void* k_pool,
               const void* v_pool, int64_t num_pages, const int32_t* block_table,
               int32_t bt_stride, int32_t num_tasks, const int32_t* kv_lens,
               const tide_dims* dims, int32_t num_splits, void* out, float* lse,
               void* workspace, size_t workspace_bytes, bool fused, bool in_scratch,
               void* stream) {
  int rc = check_dims(dims);
  if (rc != TIDE_OK) return rc;
  if (num_tasks < 0 || num_splits < 0) return TIDE_ERR_INVALID_ARG;
  if (num_tasks == 0) return TIDE_OK;
  if (num_pages <= 0 || bt_stride <= 0) return TIDE_ERR_INVALID_ARG;
  Plan plan;
  rc = make_plan(TIDE_OP_DECODE, num_tasks, kv_lens, nullptr, *dims, num_splits, bt_stride, true,
                 &plan);
  if (rc != TIDE_OK) return rc;
  if (!q || !k_pool || !v_pool || !block_table || !out) return TIDE_ERR_INVALID_ARG;
  if (fused && (!k_new || !v_new)) return TIDE_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (in_scratch) {
    if (plan.total_bytes > (size_t)TIDE_NOALLOC_SCRATCH_BYTES) return TIDE_ERR_CAPACITY;
    rc = scratch_address(&workspace);
    if (rc != TIDE_OK) return rc;
    // the blob starts with the zeroed header, so this also clears the error flags
    if (hipMemcpyAsync(workspace, plan.blob.data(), plan.blob.size(), hipMemcpyHostToDevice, s) !=
        hipSuccess)
      return TIDE_ERR_HIP;
  } else {
    if (!workspace) return TIDE_ERR_INVALID_ARG;
    if (workspace_bytes < plan.total_bytes) return TIDE_ERR_CAPACITY;
    rc = upload(plan, workspace, s);
    if (rc != TIDE_OK) return rc;
  }
  DecodeArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = block_table;
  a.num_pages = num_pages;
  a.bt_stride = bt_stride;
  a.num_q_heads = dims->num_q_heads;
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.scale_log2 = dims->sm_scale * 1.44269504088896340736f;
  a.num_tasks = num_tasks;
  a.num_items = plan.num_items;
  a.chunk = plan.chunk;
  a.max_splits = plan.max_splits;
  a.tasks = at<TaskDesc>(workspace, plan.tasks_off);
  a.items = at<DecodeItem>(workspace, plan.items_off);
  a.part_o = at_mut<float>(workspace, plan.part_o_off);
  a.part_ml = at_mut<float>(workspace, plan.part_ml_off);
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.error_flags = at_mut<int32_t>(workspace, 0);
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.tickets = plan.fold_merge ? at_mut<int32_t>(workspace, plan.tickets_off) : nullptr;
  return finish(launch_decode(a, dims->head_dim, false, s), workspace, s);
}

}  // namespace
}  // namespace tide

using namespace tide;

extern "C" {

TIDE_API int tide_workspace_size(int op, int32_t num_tasks, const int32_t* lens_a,
                                 const int32_t* lens_b, const tide_dims* dims,
                                 int32_t num_splits, size_t* bytes_out) {
  try {
    if (!bytes_out) return TIDE_ERR_INVALID_ARG;
    int rc = check_dims(dims);
    if (rc != TIDE_OK) return rc;
    Plan plan;
    rc = make_plan(op, num_tasks, lens_a, lens_b, *dims, num_splits, -1, false, &plan);
    if (rc != TIDE_OK) return rc;
    *bytes_out = plan.total_bytes;
    return TIDE_OK;
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_plan_info_get(int op, int32_t num_tasks, const int32_t* lens_a,
                               const int32_t* lens_b, const tide_dims* dims, int32_t num_splits,
                               tide_plan_info* out) {
  try {
    if (!out) return TIDE_ERR_INVALID_ARG;
    int rc = check_dims(dims);
    if (rc != TIDE_OK) return rc;
    Plan plan;
    rc = make_plan(op, num_tasks, lens_a, lens_b, *dims, num_splits, -1, false, &plan);
    if (rc != TIDE_OK) return rc;
    *out = tide_plan_info{};
    out->num_items = plan.num_items;
    out->workspace_bytes = plan.total_bytes;
    if (op == TIDE_OP_DECODE) {
      out->waves_per_group = decode_waves(plan.num_items);
      out->max_splits = plan.max_splits;
      out->merge_in_kernel = plan.fold_merge ? 1 : 0;
    } else if (op == TIDE_OP_KV_APPEND) {
      out->waves_per_group = append_waves();
    } else {
      out->waves_per_group = plan.waves;
      out->split = plan.split ? 1 : 0;
    }
    return TIDE_OK;
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_kv_append(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                            int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                            int32_t num_tasks, const int32_t* prefix_lens,
                            const int32_t* extend_lens, const tide_dims* dims, void* workspace,
                            size_t workspace_bytes, void* stream) {
  try {
    int rc = check_dims(dims);
    if (rc != TIDE_OK) return rc;
    if (num_tasks < 0) return TIDE_ERR_INVALID_ARG;
    if (num_tasks == 0) return TIDE_OK;
    if (num_pages <= 0 || bt_stride <= 0) return TIDE_ERR_INVALID_ARG;
    Plan plan;
    rc = make_plan(TIDE_OP_KV_APPEND, num_tasks, prefix_lens, extend_lens, *dims, 0, bt_stride,
                   true, &plan);
    if (rc != TIDE_OK) return rc;
    if (plan.num_items == 0) return TIDE_OK;
    if (!k_new || !v_new || !k_pool || !v_pool || !block_table || !workspace)
      return TIDE_ERR_INVALID_ARG;
    if (workspace_bytes < plan.total_bytes) return TIDE_ERR_CAPACITY;
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = upload(plan, workspace, s);
    if (rc != TIDE_OK) return rc;
    AppendArgs a;
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.k_pool = static_cast<uint16_t*>(k_pool);
    a.v_pool = static_cast<uint16_t*>(v_pool);
    a.block_table = block_table;
    a.num_pages = num_pages;
    a.bt_stride = bt_stride;
    a.num_kv_heads = dims->num_kv_heads;
    a.head_dim = dims->head_dim;
    a.num_items = plan.num_items;
    a.tasks = at<TaskDesc>(workspace, plan.tasks_off);
    a.items = at<AppendItem>(workspace, plan.items_off);
    a.error_flags = at_mut<int32_t>(workspace, 0);
    return finish(launch_kv_append(a, s), workspace, s);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_extend_attn(const void* q, const void* k_pool, const void* v_pool,
                              int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                              int32_t num_tasks, const int32_t* prefix_lens,
                              const int32_t* extend_lens, const tide_dims* dims, void* out,
                              float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    return run_extend(TIDE_OP_EXTEND, q, k_pool, v_pool, num_pages, block_table, bt_stride,
                      num_tasks, prefix_lens, extend_lens, dims, out, lse, workspace,
                      workspace_bytes, stream);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_extend_append_attn(const void* q, const void* k_new, const void* v_new,
                                     void* k_pool, void* v_pool, int64_t num_pages,
                                     const int32_t* block_table, int32_t bt_stride,
                                     int32_t num_tasks, const int32_t* prefix_lens,
                                     const int32_t* extend_lens, const tide_dims* dims, void* out,
                                     float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  try {
    return run_extend(TIDE_OP_EXTEND, q, k_pool, v_pool, num_pages, block_table, bt_stride,
                      num_tasks, prefix_lens, extend_lens, dims, out, lse, workspace,
                      workspace_bytes, stream, k_new, v_new, true);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_full_prefill_attn(const void* q, const void* k_pool, const void* v_pool,
                                    int64_t num_pages, const int32_t* block_table,
                                    int32_t bt_stride, int32_t num_tasks, const int32_t* seq_lens,
                                    const tide_dims* dims, void* out, float* lse,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  try {
    return run_extend(TIDE_OP_FULL_PREFILL, q, k_pool, v_pool, num_pages, block_table,
                      bt_stride, num_tasks, seq_lens, nullptr, dims, out, lse, workspace,
                      workspace_bytes, stream);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_decode_attn(const void* q, const void* k_pool, const void* v_pool,
                              int64_t num_pages, const int32_t* block_table, int32_t bt_stride,
                              int32_t num_tasks, const int32_t* kv_lens, const tide_dims* dims,
                              int32_t num_splits, void* out, float* lse, void* workspace,
                              size_t workspace_bytes, void* stream) {
  try {
    return run_decode(q, nullptr, nullptr, k_pool, v_pool, num_pages, block_table, bt_stride,
                      num_tasks, kv_lens, dims, num_splits, out, lse, workspace, workspace_bytes,
                      false, false, stream);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_decode_append_attn(const void* q, const void* k_new, const void* v_new,
                                     void* k_pool, void* v_pool, int64_t num_pages,
                                     const int32_t* block_table, int32_t bt_stride,
                                     int32_t num_tasks, const int32_t* kv_lens,
                                     const tide_dims* dims, int32_t num_splits, void* out,
                                     float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  try {
    return run_decode(q, k_new, v_new, k_pool, v_pool, num_pages, block_table, bt_stride,
                      num_tasks, kv_lens, dims, num_splits, out, lse, workspace, workspace_bytes,
                      true, false, stream);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_decode_attn_noalloc(const void* q, const void* k_pool, const void* v_pool,
                                      int64_t num_pages, const int32_t* block_table,
                                      int32_t bt_stride, int32_t num_tasks,
                                      const int32_t* kv_lens, const tide_dims* dims,
                                      int32_t num_splits, void* out, float* lse, void* stream) {
  try {
    return run_decode(q, nullptr, nullptr, k_pool, v_pool, num_pages, block_table, bt_stride,
                      num_tasks, kv_lens, dims, num_splits, out, lse, nullptr, 0, false, true,
                      stream);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_workspace_size_shared(int32_t num_tasks, const int32_t* kv_lens,
                                        int32_t num_groups, const int32_t* group_start,
                                        const int32_t* shared_lens, const tide_dims* dims,
                                        int32_t num_splits, size_t* bytes_out) {
  try {
    if (!bytes_out) return TIDE_ERR_INVALID_ARG;
    int rc = check_dims(dims);
    if (rc != TIDE_OK) return rc;
    Plan plan;
    rc = make_plan_shared(num_tasks, kv_lens, num_groups, group_start, shared_lens, *dims,
                          num_splits, -1, false, &plan);
    if (rc != TIDE_OK) return rc;
    *bytes_out = plan.total_bytes;
    return TIDE_OK;
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API int tide_decode_attn_shared(const void* q, const void* k_pool, const void* v_pool,
                                     int64_t num_pages, const int32_t* block_table,
                                     int32_t bt_stride, int32_t num_tasks, const int32_t* kv_lens,
                                     int32_t num_groups, const int32_t* group_start,
                                     const int32_t* shared_lens, const tide_dims* dims,
                                     int32_t num_splits, void* out, float* lse, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  try {
    int rc = check_dims(dims);
    if (rc != TIDE_OK) return rc;
    if (num_tasks < 0 || num_splits < 0) return TIDE_ERR_INVALID_ARG;
    if (num_tasks == 0) return TIDE_OK;
    if (num_pages <= 0 || bt_stride <= 0) return TIDE_ERR_INVALID_ARG;
    Plan plan;
    rc = make_plan_shared(num_tasks, kv_lens, num_groups, group_start, shared_lens, *dims,
                          num_splits, bt_stride, true, &plan);
    if (rc != TIDE_OK) return rc;
    if (!q || !k_pool || !v_pool || !block_table || !out || !workspace)
      return TIDE_ERR_INVALID_ARG;
    if (workspace_bytes < plan.total_bytes) return TIDE_ERR_CAPACITY;
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = upload(plan, workspace, s);
    if (rc != TIDE_OK) return rc;
    DecodeArgs a;
    a.q = static_cast<const uint16_t*>(q);
    a.k_pool = static_cast<const uint16_t*>(k_pool);
    a.v_pool = static_cast<const uint16_t*>(v_pool);
    a.block_table = block_table;
    a.num_pages = num_pages;
    a.bt_stride = bt_stride;
    a.num_q_heads = dims->num_q_heads;
    a.num_kv_heads = dims->num_kv_heads;
    a.group = dims->num_q_heads / dims->num_kv_heads;
    a.scale_log2 = dims->sm_scale * 1.44269504088896340736f;
    a.num_tasks = num_tasks;
    a.num_items = plan.num_items;
    a.chunk = plan.chunk;
    a.max_splits = plan.max_splits;
    a.tasks = at<TaskDesc>(workspace, plan.tasks_off);
    a.items = at<SharedDecodeItem>(workspace, plan.items_off);
    a.part_o = at_mut<float>(workspace, plan.part_o_off);
    a.part_ml = at_mut<float>(workspace, plan.part_ml_off);
    a.out = static_cast<uint16_t*>(out);
    a.lse = lse;
    a.error_flags = at_mut<int32_t>(workspace, 0);
    a.k_new = nullptr;
    a.v_new = nullptr;
    a.tickets = nullptr;
    return finish(launch_decode(a, dims->head_dim, true, s), workspace, s);
  } catch (...) {
    return TIDE_ERR_HIP;
  }
}

TIDE_API const char* tide_status_string(int status) {
  switch (status) {
    case TIDE_OK: return "ok";
    case TIDE_ERR_INVALID_ARG: return "invalid argument";
    case TIDE_ERR_UNSUPPORTED: return "unsupported shape";
    case TIDE_ERR_CAPACITY: return "capacity exceeded (block table or workspace too small)";
    case TIDE_ERR_HIP: return "HIP runtime error";
    case TIDE_ERR_PAGE_RANGE: return "block-table page id out of range";
    default: return "unknown status";
  }
}

TIDE_API void tide_shutdown(void) {
  std::lock_guard<std::mutex> lock(g_mutex);
  for (DeviceStaging* ds : g_staging) {
    if (!ds) continue;
    for (StagingSlot& s : ds->slots) {
      if (s.pending) (void)wait_slot(s);
      if (s.host) (void)hipHostFree(s.host);
      if (s.flags) (void)hipHostFree(s.flags);
    }
    delete ds;
  }
  g_staging.clear();
}

}  // extern "C"
