// KV-append: store new tokens' K/V into their pages of the shared pool -- the state
// Continuous Task Batching keeps resident so that a resumed task need not recompute
// its history (TideRL Section 4).  Position p of a task lives in page BT[p / 16],
// slot p % 16; K and V pages are both [16 slots][d], so a token's row of either is one
// contiguous run of d values and the append is a plain copy.
//
// One wave per (task, logical page, kv head).  Rows are copied in 16-byte pieces.  A
// page this append fills is copied with every lane's loads issued before any store
// (the compiler cannot rule out aliasing between the new rows and the pool, and would
// otherwise wait for each load before the next); a page only partly appended takes
// exactly its new slots, so it keeps its other slots.
#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWaves = 4;

template <int D>
__global__ __launch_bounds__(kWaves * 64) void kv_append_kernel(AppendArgs a) {
  constexpr int kG = D / 8;  // 16-byte pieces per row
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.y * kWaves + wave;
  const AppendItem it = a.items[blockIdx.x];
  const TaskDesc td = a.tasks[it.task];
  const int32_t phys = a.block_table[(int64_t)it.task * a.bt_stride + it.lpage];
  const bool page_ok = phys >= 0 && phys < a.num_pages;
  if (!page_ok && threadIdx.x == 0) atomicOr(a.error_flags, 1);
  if (g >= a.num_kv_heads || !page_ok) return;

  const int s0 = it.pos_begin % kPage;
  const int n = it.pos_end - it.pos_begin;
  const int64_t row0 = (int64_t)td.row_start + (it.pos_begin - td.prefix);
  const int64_t blk = ((int64_t)phys * a.num_kv_heads + g) * (int64_t)(kPage * D);

  if (n == kPage) {
    constexpr int kPer = kPage * kG / 64;
    u32x4 kk[kPer], vv[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = lane + 64 * i, sl = idx / kG, part = idx % kG;
      const int64_t src = ((row0 + sl) * a.num_kv_heads + g) * D + part * 8;
      kk[i] = load_u32x4(a.k_new + src);
      vv[i] = load_u32x4(a.v_new + src);
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = lane + 64 * i;  // slot idx / kG, piece idx % kG: blk + 8 * idx
      store_u32x4(a.k_pool + blk + 8 * idx, kk[i]);
      store_u32x4(a.v_pool + blk + 8 * idx, vv[i]);
    }
  } else {
    for (int idx = lane; idx < n * kG; idx += 64) {
      const int sl = idx / kG, part = idx % kG;
      const int64_t src = ((row0 + sl) * a.num_kv_heads + g) * D + part * 8;
      const int64_t dst = blk + (int64_t)(s0 + sl) * D + part * 8;
      store_u32x4(a.k_pool + dst, load_u32x4(a.k_new + src));
      store_u32x4(a.v_pool + dst, load_u32x4(a.v_new + src));
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

int append_waves() { return kern::kWaves; }

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (a.head_dim == 128) return kern::launch<128>(a, stream);
  if (a.head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
