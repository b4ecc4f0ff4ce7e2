// Extend attention with the KV-append of the new tokens fused in: the instantiations of
// the kernel in attn_extend.h that read keys at or past each task's prefix straight from
// the new rows and write those rows into the pool (tide_extend_append_attn).  Compiled
// apart from the plain variants so that the two build in parallel; the split-KV merge is
// launched by attn_extend.hip.
#include "attn_extend.h"

namespace tide {
namespace kern {

template <int D, bool kSplit>
hipError_t launch_attn_append(const ExtendArgs& a, hipStream_t stream) {
  if (a.lse)
    hipLaunchKernelGGL((extend_attn_kernel<D, true, kSplit, true>), dim3(a.num_items),
                       dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((extend_attn_kernel<D, false, kSplit, true>), dim3(a.num_items),
                       dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template __global__ void extend_attn_kernel<128, false, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<128, false, true, true>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, true, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, true, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, true, true>(ExtendArgs);

hipError_t launch_extend_append_attn(const ExtendArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 128)
    return a.chunk_items ? launch_attn_append<128, true>(a, stream) : launch_attn_append<128, false>(a, stream);
  if (head_dim == 64)
    return a.chunk_items ? launch_attn_append<64, true>(a, stream) : launch_attn_append<64, false>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace kern
}  // namespace tide
