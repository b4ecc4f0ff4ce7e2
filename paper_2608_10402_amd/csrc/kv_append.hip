// KV-append: store new tokens' K/V into their pages of the shared pool -- the state
// Continuous Task Batching keeps resident so that a resumed task need not recompute
// its history (TideRL Section 4).  Position p of a task lives in page BT[p / 16],
// slot p % 16.  K pages are [16 slots][d]; V pages are stored transposed, [d][16 slots],
// so that attention reads V^T operands with plain 16-byte loads.
//
// One wave per (task, logical page, kv head).  K rows are copied with 16-byte loads and
// stores.  V rows are staged in LDS and written back transposed: a page filled by this
// append takes 16-byte stores (half a head-dim row of 8 slots each); a page that is only
// partly appended takes 2-byte stores of exactly its new slots, consecutive lanes
// covering consecutive slots of one head-dim row, so it keeps its other slots.
#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWaves = 4;

template <int D>
__global__ __launch_bounds__(kWaves * 64) void kv_append_kernel(AppendArgs a) {
  constexpr int kPitch = D + 2;  // odd word pitch: column reads hit distinct banks
  __shared__ uint16_t v_lds[kWaves][kPage * kPitch];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.y * kWaves + wave;
  const AppendItem it = a.items[blockIdx.x];
  const TaskDesc td = a.tasks[it.task];
  const int32_t phys = a.block_table[(int64_t)it.task * a.bt_stride + it.lpage];
  const bool page_ok = phys >= 0 && phys < a.num_pages;
  const bool active = g < a.num_kv_heads && page_ok;
  if (!page_ok && threadIdx.x == 0) atomicOr(a.error_flags, 1);

  const int s0 = it.pos_begin % kPage;
  const int n = it.pos_end - it.pos_begin;
  const int64_t row0 = (int64_t)td.row_start + (it.pos_begin - td.prefix);
  const int64_t blk = ((int64_t)(active ? phys : 0) * a.num_kv_heads + g) * (int64_t)(kPage * D);
  uint16_t* vl = v_lds[wave];

  if (active && n == kPage) {
    // Full page: every lane issues all its loads (kPage * D / 8 / 64 K and V pieces)
    // before any store, so they are in flight together.
    constexpr int kPer = kPage * (D / 8) / 64;
    u32x4 kk[kPer], vv[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = lane + 64 * i, sl = idx / (D / 8), part = idx % (D / 8);
      const int64_t src = ((row0 + sl) * a.num_kv_heads + g) * D + part * 8;
      kk[i] = load_u32x4(a.k_new + src);
      vv[i] = load_u32x4(a.v_new + src);
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = lane + 64 * i, sl = idx / (D / 8), part = idx % (D / 8);
      store_u32x4(a.k_pool + blk + sl * D + part * 8, kk[i]);
      uint32_t* dst = reinterpret_cast<uint32_t*>(vl + sl * kPitch + part * 8);
#pragma unroll
      for (int w = 0; w < 4; ++w) dst[w] = vv[i][w];
    }
  } else if (active) {
    for (int idx = lane; idx < n * (D / 8); idx += 64) {
      const int sl = idx / (D / 8), part = idx % (D / 8);
      const int64_t src = ((row0 + sl) * a.num_kv_heads + g) * D + part * 8;
      store_u32x4(a.k_pool + blk + (s0 + sl) * D + part * 8, load_u32x4(a.k_new + src));
      const u32x4 vv = load_u32x4(a.v_new + src);
      uint32_t* dst = reinterpret_cast<uint32_t*>(vl + (s0 + sl) * kPitch + part * 8);
#pragma unroll
      for (int w = 0; w < 4; ++w) dst[w] = vv[w];
    }
  }
  __syncthreads();
  if (active && n == kPage) {
    // Full page: each V^T row (16 slots, 32 bytes) is two 16-byte stores, one per half.
    for (int idx = lane; idx < D * 2; idx += 64) {
      const int d = idx >> 1, h = idx & 1;
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)vl[(8 * h + 2 * e) * kPitch + d] |
               ((uint32_t)vl[(8 * h + 2 * e + 1) * kPitch + d] << 16);
      store_u32x4(a.v_pool + blk + d * kPage + 8 * h, w);
    }
  } else if (active) {
    for (int idx = lane; idx < D * kPage; idx += 64) {
      const int d = idx / kPage, s = idx % kPage;
      if (s >= s0 && s < s0 + n) a.v_pool[blk + d * kPage + s] = vl[s * kPitch + d];
    }
  }
}

template <int D>
hipError_t launch(const AppendArgs& a, hipStream_t stream) {
  dim3 grid(a.num_items, (a.num_kv_heads + kWaves - 1) / kWaves);
  hipLaunchKernelGGL((kv_append_kernel<D>), grid, dim3(kWaves * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace kern

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (a.head_dim == 128) return kern::launch<128>(a, stream);
  if (a.head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
