// Host-side launchers of the gfx950 kernels (one per .hip file).
#pragma once

#include <hip/hip_runtime.h>

#include "tide_common.h"

namespace tide {

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream);
// Extend / prefill attention; with a.k_new set, the variant with the KV-append fused in.
hipError_t launch_extend(const ExtendArgs& a, int head_dim, int waves, hipStream_t stream);
namespace kern {
// The fused-append attention kernel alone (attn_extend_append.hip); launch_extend adds
// the split-KV merge.
hipError_t launch_extend_append_attn(const ExtendArgs& a, int head_dim, hipStream_t stream);
}  // namespace kern
hipError_t launch_decode(const DecodeArgs& a, int head_dim, bool shared, hipStream_t stream);
// Waves per workgroup the decode split kernel and the append kernel launch with.
int decode_waves(int32_t num_items);
int append_waves();

}  // namespace tide
