// Extend attention (and full prefill) launchers, the split-KV merge kernel, and the
// instantiations of the kernel in attn_extend.h without the fused KV-append.
#include "attn_extend.h"

namespace tide {
namespace kern {

constexpr int kMergeWaves = 4;

// One wave per (packed row, query head) of a split-KV call: combines the row's chunk
// partials; rows that were not split were written by the attention kernel.
template <int D>
__global__ __launch_bounds__(kMergeWaves * 64) void extend_merge_kernel(ExtendArgs a) {
  // wave-uniform and 32-bit (the launch has total_rows * Hq < 2^31 waves)
  const int wi = (int)blockIdx.x * kMergeWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wi >= a.total_rows * a.num_q_heads) return;
  const int row = wi / a.num_q_heads;
  const int head = wi - row * a.num_q_heads;
  const int64_t w = wi;
  const MergeRow mr = a.merge_rows[row];
  if (mr.nsplit == 0) return;
  const int64_t s0 = (int64_t)mr.base * a.num_q_heads + head;
  const int64_t ss = (int64_t)mr.stride * a.num_q_heads;
  merge_partials<D>(a.part_ml + s0 * 4, ss * 4, a.part_o + s0 * D, ss * D, mr.nsplit,
                    a.out + w * D, a.lse ? a.lse + w : nullptr);
}

template <int D, bool kSplit>
hipError_t launch_attn(const ExtendArgs& a, hipStream_t stream) {
  if (a.lse)
    hipLaunchKernelGGL((extend_attn_kernel<D, true, kSplit, false>), dim3(a.num_items),
                       dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((extend_attn_kernel<D, false, kSplit, false>), dim3(a.num_items),
                       dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch(const ExtendArgs& a, hipStream_t stream) {
  hipError_t e;
  if (a.k_new)  // the fused-append variants are compiled in attn_extend_append.hip
    e = launch_extend_append_attn(a, D, stream);
  else
    e = a.chunk_items ? launch_attn<D, true>(a, stream) : launch_attn<D, false>(a, stream);
  if (e != hipSuccess || !a.chunk_items || !a.merge_rows) return e;
  const int64_t waves = (int64_t)a.total_rows * a.num_q_heads;
  if (waves >= INT32_MAX - kMergeWaves) return hipErrorInvalidValue;
  const int blocks = (int)((waves + kMergeWaves - 1) / kMergeWaves);
  hipLaunchKernelGGL((extend_merge_kernel<D>), dim3(blocks), dim3(kMergeWaves * 64), 0, stream, a);
  return hipGetLastError();
}

// Every variant is instantiated explicitly: the host pass otherwise emits the launch stub
// of only one of the specialisations that differ in a bool.
template __global__ void extend_attn_kernel<128, false, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, false, true, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, true, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, true, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, true, false>(ExtendArgs);

}  // namespace kern

hipError_t launch_extend(const ExtendArgs& a, int head_dim, int waves, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (waves != kern::kWaves) return hipErrorInvalidValue;
  if (head_dim == 128) return kern::launch<128>(a, stream);
  if (head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
