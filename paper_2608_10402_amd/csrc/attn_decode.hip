// Decode attention over the paged KV pool: one query token per task (the action tokens
// a task generates between environment turns, TideRL Section 2.1) against its whole
// retained context.  The context is split into chunks processed in parallel and merged
// by log-sum-exp weights (split-K, as in Flash-Decoding, Dao et al. 2023).
//
// Decode reads every K/V byte of the context once and does ~2 flops per byte, so it is
// bound by HBM bandwidth.  The design therefore minimises everything but the stream:
//   * One wave per (task, kv head, chunk).  The G query heads of the kv head share every
//     K/V load; they are the columns of v_mfma_f32_16x16x32_bf16 (G <= 16), so the
//     contraction costs a few MFMA issues per 2 KB loaded and no VALU dot products.
//   * Shared-prefix variant (a GRPO group's trajectories share their task's prompt pages,
//     TideRL Section 2.1; CTB keeps them on one rank, Section 4.2): a chunk of the shared
//     prefix is one wave for several trajectories, whose (trajectory, head) pairs fill the
//     16 MFMA columns, so the prefix is read once per group of trajectories instead of
//     once per trajectory.  Each trajectory's own keys are ordinary chunks; all of them are
//     splits of the same merge.
//   * Operands go straight from HBM into MFMA registers (no LDS): for S^T = K.Q^T a lane
//     loads 16 contiguous bytes of one key row; for O^T += V^T.P^T it loads two 8-byte
//     pieces of transposed V pages (4 consecutive token slots of one head-dim entry in
//     each page).  The S^T rows of page t are its token slots, so each lane's
//     probabilities are exactly those slots and P never moves between lanes.
//   * Every load instruction reads one page: the page block is a scalar base, lanes add
//     a fixed offset.  Page ids arrive 64 at a time (one vector load, then readlane).
//   * Two register buffers in ping-pong keep the next 32-key step in flight; at most
//     256 registers so two waves share each SIMD.
//   * Partial (o, m, l) per split go to the workspace; a second small kernel merges them.
#include <type_traits>

#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWavesPerBlock = 4;

// One 32-key step (pages p0 = keys k..k+15 and p1 = k+16..k+31) in registers.
//   k[t][c]: S^T operand for page t, head-dim chunk c (MFMA row = token slot)
//   v[t][h]: V^T operand halves for head-dim tile t: slots 4*grp..4*grp+3 of page h
template <int D>
struct DecodeRegs {
  u32x4 k[2][D / 32];
  uint2 v[D / 16][2];
};

// Buffer resource of one (page, kv head) block: base in SGPRs, range = the block, so each
// load is a 32-bit lane offset plus an immediate (raw buffer, gfx9 descriptor format).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t block_rsrc(const uint8_t* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), 0, bytes, 0x00020000);
}

// Cache policy of the K/V loads.  Keys that one wave alone reads (a task's context in
// plain decode, a trajectory's own keys after a shared prompt) are streamed with the
// non-temporal hint (the nt bit, aux bit 1 on gfx950): streaming reads measured 7.1 TB/s
// on MI355X with it against 6.3 TB/s without.  A shared prompt chunk, which the waves of
// a group's other subgroups read right after, keeps the default policy so that those
// reads hit L2.
constexpr int kStreamPolicy = 2;
constexpr int kSharedPolicy = 0;

// Loads of one step.  Every instruction reads a single page block.
template <int D, int kPolicy>
__device__ __forceinline__ void load_step(DecodeRegs<D>& r, __amdgpu_buffer_rsrc_t k0,
                                          __amdgpu_buffer_rsrc_t k1, __amdgpu_buffer_rsrc_t v0,
                                          __amdgpu_buffer_rsrc_t v1, uint32_t k_off,
                                          uint32_t v_off) {
#pragma unroll
  for (int c = 0; c < D / 32; ++c) {
    r.k[0][c] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(k0, k_off + 64 * c, 0, kPolicy));
    r.k[1][c] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(k1, k_off + 64 * c, 0, kPolicy));
  }
#pragma unroll
  for (int t = 0; t < D / 16; ++t) {
    r.v[t][0] = __builtin_bit_cast(
        uint2, __builtin_amdgcn_raw_buffer_load_b64(v0, v_off + 512 * t, 0, kPolicy));
    r.v[t][1] = __builtin_bit_cast(
        uint2, __builtin_amdgcn_raw_buffer_load_b64(v1, v_off + 512 * t, 0, kPolicy));
  }
}

// Keep only the first n (0..4) bf16 elements of an 8-byte V^T piece.
__device__ __forceinline__ uint2 keep_first4(uint2 x, int n) {
  uint2 r;
  r.x = x.x & ((n > 0 ? 0x0000FFFFu : 0u) | (n > 1 ? 0xFFFF0000u : 0u));
  r.y = x.y & ((n > 2 ? 0x0000FFFFu : 0u) | (n > 3 ? 0xFFFF0000u : 0u));
  return r;
}

// kShared: the items are SharedDecodeItem: keys of a prefix shared by ntasks tasks (the
// MFMA columns are then (task, query head) pairs, ntasks * G <= 16, so every K/V byte is
// loaded once for all of them), or a task's own keys after it.  Otherwise DecodeItem.
// kAppend (plain items only): the newest token of each task (position kv_len - 1) is not
// in the pool yet.  The split that holds it first writes that token's K/V from
// a.k_new / a.v_new into its pool slot, waits for the stores, then reads as usual.  No
// other split reads that slot, so the result equals appending first and then decoding.
template <int D, bool kShared, bool kAppend>
__global__ __launch_bounds__(kWavesPerBlock * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_split_kernel(DecodeArgs a) {
  const int lane = threadIdx.x & 63;
  // the wave index is uniform across the wave: say so, so the item and every address
  // derived from it stay scalar
  const int item_id = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item_id >= a.num_items) return;  // whole wave exits; no block-level barrier below
  int first_task, ntasks, kv_head, split, kbeg, kend;
  if constexpr (kShared) {
    const SharedDecodeItem it = static_cast<const SharedDecodeItem*>(a.items)[item_id];
    first_task = it.first_task;
    ntasks = it.ntasks;
    kv_head = it.kv_head;
    split = it.split;
    kbeg = it.k_begin;
    kend = it.k_end;
  } else {
    const DecodeItem it = static_cast<const DecodeItem*>(a.items)[item_id];
    first_task = it.task;
    ntasks = 1;
    kv_head = it.kv_head;
    split = it.split;
    kbeg = it.k_begin;
  }
  const TaskDesc td = a.tasks[first_task];
  const int kv_len = td.prefix + td.extend;
  if constexpr (!kShared) kend = min(kv_len, kbeg + a.chunk);
  const int npages = (kv_len + kPage - 1) / kPage;
  const int32_t* bt_row = a.block_table + (int64_t)first_task * a.bt_stride;
  const int G = a.group;
  const int col = lane & 15, grp = lane >> 4;
  const int kv_h = kv_head;
  const uint8_t* kpool = reinterpret_cast<const uint8_t*>(a.k_pool);
  const uint8_t* vpool = reinterpret_cast<const uint8_t*>(a.v_pool);
  constexpr int64_t kBlk = (int64_t)kPage * D * 2;  // bytes of one (page, kv head) block

  // Column col: task first_task + col / G, query head kv_head * G + col % G (no column
  // past ntasks * G: its Q is zero and nothing is written for it)
  const bool col_ok = col < ntasks * G;
  const int ctask = kShared ? first_task + col / G : first_task;
  const int chead = kShared ? col % G : col;
  const int crow = kShared ? (col_ok ? a.tasks[ctask].row_start : 0) : td.row_start;
  bf16x8 qf[D / 32];
  const int64_t qrow = (int64_t)crow * a.num_q_heads + kv_h * G + chead;
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
    qf[c] = as_bf16x8(col_ok ? load_u32x4(a.q + qrow * D + 32 * c + 8 * grp) : zero_u32x4());

  const uint32_t k_off = (uint32_t)(col * D * 2 + 16 * grp);       // token slot `col`
  const uint32_t v_off = (uint32_t)(col * kPage * 2 + 8 * grp);    // head-dim row `col`

  // Page ids of this split, 64 at a time: lane i holds logical page lp0 + i.
  int lp_batch = -1;
  int32_t pid = 0;
  bool flag_error = false;  // an invalid page id was seen (reported once, at the end)
  auto page_block = [&](int lp) -> int64_t {
    if (lp - lp_batch >= 64 || lp_batch < 0) {
      lp_batch = lp;
      const int mine = lp + lane;
      pid = mine < npages ? bt_row[mine] : 0;
    }
    const int32_t p = __builtin_amdgcn_readlane(pid, lp - lp_batch);
    const bool bad = p < 0 || p >= a.num_pages || lp >= npages;
    // pages past the context (and invalid ids) read page 0: masked / zeroed below
    const int64_t blk = ((int64_t)(bad ? 0 : p) * a.num_kv_heads + kv_h) * kBlk;
    if (bad && lp < npages) flag_error = true;
    return blk;
  };
  auto load = [&](DecodeRegs<D>& r, int k, auto policy_tag) {
    const int64_t b0 = page_block(k / kPage), b1 = page_block(k / kPage + 1);
    load_step<D, decltype(policy_tag)::value>(
        r, block_rsrc(kpool + b0, (int)kBlk), block_rsrc(kpool + b1, (int)kBlk),
        block_rsrc(vpool + b0, (int)kBlk), block_rsrc(vpool + b1, (int)kBlk), k_off, v_off);
  };

  f32x4 o[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t) o[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;

  auto compute = [&](DecodeRegs<D>& cur, int k) {
    // S^T for page t: s[t][e] is key k + 16*t + 4*grp + e of query head `col`
    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < D / 32; ++c) s[t] = mfma16(as_bf16x8(cur.k[t][c]), qf[c], s[t]);
    }
    // keys at or past kend (the context's end, or the shared prefix's) are not this item's
    const bool tail = k + 2 * kPage > kend;
    float mt = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float x = s[t][e] * a.scale_log2;
        if (tail) x = (k + 16 * t + 4 * grp + e < kend) ? x : -INFINITY;
        s[t][e] = x;
        mt = fmaxf(mt, x);
      }
    if (tail) {  // V slots past kend must not reach the MFMA (NaN * 0 = NaN)
#pragma unroll
      for (int t = 0; t < D / 16; ++t)
#pragma unroll
        for (int hp = 0; hp < 2; ++hp)
          cur.v[t][hp] = keep_first4(cur.v[t][hp], kend - (k + 16 * hp + 4 * grp));
    }
    mt = fmaxf(mt, xor_shfl(mt, 16));
    mt = fmaxf(mt, xor_shfl(mt, 32));
    if (__any(mt > m_ref + kRescaleSlack)) {
      const float m_new = fmaxf(m_ref, mt);
      const float alpha = fast_exp2(m_ref - m_new);
      l_part *= alpha;
      l_exact *= alpha;
#pragma unroll
      for (int t = 0; t < D / 16; ++t) o[t] *= alpha;
      m_ref = m_new;
    }
    // P^T operand: slots 0..3 = page 0 keys 4*grp.., slots 4..7 = page 1 keys 4*grp..
    u32x4 w;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float p0 = fast_exp2(s[t][2 * e] - m_ref);
        const float p1 = fast_exp2(s[t][2 * e + 1] - m_ref);
        w[2 * t + e] = pack_bf16x2(p0, p1);
        l_part = add_bf16x2(w[2 * t + e], l_part);
        l_exact += p0 + p1;
      }
    const bf16x8 pb = as_bf16x8(w);
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
      const u32x4 vv = {cur.v[t][0].x, cur.v[t][0].y, cur.v[t][1].x, cur.v[t][1].y};
      o[t] = mfma16(as_bf16x8(vv), pb, o[t]);
    }
  };

  if constexpr (kAppend) {
    // The split that ends the context appends its newest token before reading: K row
    // and V^T column of slot pos % 16, then waits until the stores have completed, so
    // the loads below return them.  No other wave reads this page (splits end on
    // 32-key boundaries), and no earlier load in this kernel can have put a stale copy
    // of it in this CU's L1.
    if (kend == kv_len) {
      const int pos = kv_len - 1, slot = pos % kPage;
      const int32_t p = bt_row[pos / kPage];
      if (p >= 0 && p < a.num_pages) {
        const int64_t row = (int64_t)td.row_start * a.num_kv_heads + kv_h;
        const int64_t blk = ((int64_t)p * a.num_kv_heads + kv_h) * (int64_t)(kPage * D);
        uint16_t* kdst = const_cast<uint16_t*>(a.k_pool) + blk + (int64_t)slot * D;
        uint16_t* vdst = const_cast<uint16_t*>(a.v_pool) + blk + slot;
        const uint16_t* kn = a.k_new + row * D;
        const uint16_t* vn = a.v_new + row * D;
        if (lane < D / 8) store_u32x4(kdst + 8 * lane, load_u32x4(kn + 8 * lane));
#pragma unroll
        for (int d = lane; d < D; d += 64) vdst[d * kPage] = vn[d];
      } else {
        flag_error = true;
      }
      __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) expcnt(0) lgkmcnt(0): stores done
      __atomic_signal_fence(__ATOMIC_SEQ_CST);  // and no load is moved above them
    }
  }

  // Two register buffers in ping-pong: the next step is in flight while one is used.
  auto stream = [&](auto policy_tag) {
    DecodeRegs<D> ra, rb;
    load(ra, kbeg, policy_tag);
    for (int k = kbeg; k < kend; k += 2 * kDecodeStep) {
      if (k + kDecodeStep < kend) load(rb, k + kDecodeStep, policy_tag);
      compute(ra, k);
      if (k + kDecodeStep >= kend) break;
      if (k + 2 * kDecodeStep < kend) load(ra, k + 2 * kDecodeStep, policy_tag);
      compute(rb, k + kDecodeStep);
    }
  };
  if (kShared && ntasks > 1)
    stream(std::integral_constant<int, kSharedPolicy>());
  else
    stream(std::integral_constant<int, kStreamPolicy>());

  if (flag_error && lane == 0) atomicOr(a.error_flags, 1);
  float l_tot = l_part + xor_shfl(l_part, 16);
  l_tot += xor_shfl(l_tot, 32);
  float l_ex = l_exact + xor_shfl(l_exact, 16);
  l_ex += xor_shfl(l_ex, 32);
  if (col_ok) {
    const int64_t slot =
        ((int64_t)ctask * a.num_q_heads + kv_h * G + chead) * a.max_splits + split;
    float* po = a.part_o + slot * D;
#pragma unroll
    for (int t = 0; t < D / 16; ++t)
      *reinterpret_cast<f32x4*>(po + 16 * t + 4 * grp) = o[t];
    if (grp == 0) {
      f32x4 ml = {m_ref, l_tot, l_ex, 0.0f};
      *reinterpret_cast<f32x4*>(a.part_ml + slot * 4) = ml;
    }
  }
}

// One wave per (task, query head): combine the task's split partials.
template <int D>
__global__ __launch_bounds__(kWavesPerBlock * 64) void decode_merge_kernel(DecodeArgs a) {
  // wave-uniform and 32-bit (the launch has num_tasks * Hq < 2^31 waves)
  const int row = (int)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= a.num_tasks * a.num_q_heads) return;
  const int task = row / a.num_q_heads;
  const int64_t r = row;
  merge_partials<D>(a.part_ml + r * a.max_splits * 4, 4, a.part_o + r * a.max_splits * D, D,
                    a.tasks[task].aux, a.out + r * D, a.lse ? a.lse + r : nullptr);
}

template <int D, bool kShared, bool kAppend>
hipError_t launch(const DecodeArgs& a, hipStream_t stream) {
  if (a.num_items > 0) {
    const int blocks = (a.num_items + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((decode_split_kernel<D, kShared, kAppend>), dim3(blocks),
                       dim3(kWavesPerBlock * 64), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t rows = (int64_t)a.num_tasks * a.num_q_heads;
  if (rows >= INT32_MAX - kWavesPerBlock) return hipErrorInvalidValue;
  if (rows > 0) {
    const int blocks = (int)((rows + kWavesPerBlock - 1) / kWavesPerBlock);
    hipLaunchKernelGGL((decode_merge_kernel<D>), dim3(blocks), dim3(kWavesPerBlock * 64), 0,
                       stream, a);
  }
  return hipGetLastError();
}

// Both variants of each head size are instantiated explicitly: the host pass otherwise
// emits the launch stub of only one of two specialisations that differ in the bool.
template __global__ void decode_split_kernel<128, false, false>(DecodeArgs);
template __global__ void decode_split_kernel<128, true, false>(DecodeArgs);
template __global__ void decode_split_kernel<128, false, true>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, false>(DecodeArgs);
template __global__ void decode_split_kernel<64, true, false>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, true>(DecodeArgs);

}  // namespace kern

hipError_t launch_decode(const DecodeArgs& a, int head_dim, bool shared, hipStream_t stream) {
  const bool append = a.k_new != nullptr;
  if (shared && append) return hipErrorInvalidValue;
  if (head_dim == 128) {
    if (shared) return kern::launch<128, true, false>(a, stream);
    return append ? kern::launch<128, false, true>(a, stream) : kern::launch<128, false, false>(a, stream);
  }
  if (head_dim == 64) {
    if (shared) return kern::launch<64, true, false>(a, stream);
    return append ? kern::launch<64, false, true>(a, stream) : kern::launch<64, false, false>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace tide
