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
//   * K and V pages are both loaded in whole 128-byte lines.  The S^T = K.Q^T operand
//     needs 16 key rows x 16 bytes per instruction, so loading it directly would read 16
//     half cache lines per instruction; HBM streams such a pattern about 14% slower than
//     whole lines.  Instead each wave copies its K pages into its own LDS region with
//     direct-to-LDS buffer loads (8 rows x 128 bytes per instruction) and reads the
//     operand with ds_read_b128 from an XOR-swizzled layout that keeps the 16 rows of one
//     read in distinct banks.  V pages ([16 slots][d], like K) are loaded into registers,
//     1 KB of contiguous rows per instruction; once the step's scores are computed, the
//     wave writes them over its K copy in LDS and reads the O^T += V^T.P^T operands back
//     with ds_read_b64_tr_b16, which transposes 4 key rows x 16 head-dim entries across
//     each 16-lane group.  The S^T rows of page t are its token slots, so each lane's
//     probabilities are exactly those slots and P never moves between lanes.
//   * Every load instruction reads one page: the page block is a scalar base, lanes add
//     a fixed offset.  Page ids come from scalar loads.
//   * Two buffers in ping-pong (LDS for K, registers for V) keep the next 32-key step in
//     flight; at most 256 registers and 16 KB of LDS per wave, so two waves share each
//     SIMD.  A large launch runs 8-wave workgroups (8 consecutive items onto one CU), a
//     small one 4-wave workgroups.
//   * Partial (o, m, l) per split go to the workspace; a second small kernel merges them.
#include <type_traits>

#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

// Waves per workgroup of the split kernel: 8 consecutive items (at 8 kv heads, all heads
// of one task's chunk, whose page blocks are contiguous) on one CU when the launch has
// enough items to give every CU a full workgroup; otherwise 4, so that a small launch
// still spreads over all CUs (a 4-wave workgroup takes half a CU's LDS).
constexpr int kBigWaves = 8, kSmallWaves = 4;
constexpr int kBigLaunchItems = 2048;  // 256 CUs x 8 waves
constexpr int kMergeWaves = 4;

// V of one 32-key step (pages p0 = keys k..k+15 and p1 = k+16..k+31): v[h][i] is this
// lane's 16 bytes of load i of page h, which covers page bytes 1024 i .. 1024 i + 1023.
// The step's K pages sit in a per-wave LDS buffer.
template <int D>
struct DecodeRegs {
  static constexpr int kLoads = kPage * D * 2 / 1024;  // 1 KB loads per page
  u32x4 v[2][kLoads];
};

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// V page layout in LDS, written over the step's K copy once its scores are computed: row
// r (16 of them, 2D bytes each) keeps its order, and its 32-byte blocks are XOR-swizzled
// by vsw(r), so that the 8 rows x 32 bytes a half-wave reads with ds_read_b64_tr_b16 fall
// in distinct banks, and the 16 lanes of a 16-byte write of one row too.
template <int D>
struct VLds {
  static constexpr int kNG = D / 8;  // 16-byte granules per row
  static __device__ __forceinline__ int vsw(int r) { return D == 128 ? (r & 7) : ((r >> 1) & 3); }
  // byte offset, inside a page copy, of 16-byte granule g of row r
  static __device__ __forceinline__ uint32_t offset(int r, int g) {
    return (uint32_t)(r * 2 * D + 32 * ((g >> 1) ^ vsw(r)) + 16 * (g & 1));
  }
};

// K page layout in LDS.  A page block is 16 key rows of D bf16 (2D bytes = D/8 granules
// of 16 bytes).  It is copied by 2 * (D/64) direct-to-LDS instructions; instruction
// i = a * (D/64) + h covers rows 8a..8a+7 and granules 8h..8h+7 of each, lane l taking
// row r = 8a + l/8 and granule 8h + ((l%8) ^ ((r/2)%8)), which lands at byte
// 1024 * i + 16 * l of the page's LDS copy.  Granule g of row r is therefore found at
// slot 8 * (r%8) + ((g%8) ^ ((r/2)%8)) of instruction (r/8) * (D/64) + g/8; a read of one
// granule by the 16 rows of an MFMA operand touches 16 distinct 16-byte bank groups.
template <int D>
struct KLds {
  static constexpr int kHalves = D / 64;           // 128-byte halves of a key row
  static constexpr int kDma = 2 * kHalves;         // direct-to-LDS loads per page
  static constexpr int kPageBytes = kPage * D * 2;
  static_assert(kDma * 1024 == kPageBytes, "page = whole 1 KB loads");
  // global byte offset, inside the page block, of lane `lane`'s 16 bytes in load i
  static __device__ __forceinline__ uint32_t src_offset(int i, int lane) {
    const int r = 8 * (i / kHalves) + (lane >> 3);
    const int g = 8 * (i % kHalves) + ((lane & 7) ^ ((r >> 1) & 7));
    return (uint32_t)(r * 2 * D + 16 * g);
  }
  // LDS byte offset, inside the page copy, of granule g of row r
  static __device__ __forceinline__ uint32_t lds_offset(int r, int g) {
    const int i = (r >> 3) * kHalves + (g >> 3);
    return (uint32_t)(1024 * i + 16 * (8 * (r & 7) + ((g & 7) ^ ((r >> 1) & 7))));
  }
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

// Loads of one step.  Every instruction reads a single page block: the K pages go to
// kbuf (page t at t * kPageBytes), the V rows to registers.
template <int D, int kPolicy>
__device__ __forceinline__ void load_step(DecodeRegs<D>& r, uint8_t* kbuf,
                                          __amdgpu_buffer_rsrc_t k0, __amdgpu_buffer_rsrc_t k1,
                                          __amdgpu_buffer_rsrc_t v0, __amdgpu_buffer_rsrc_t v1,
                                          const uint32_t (&k_src)[KLds<D>::kDma],
                                          uint32_t v_off) {
  using L = KLds<D>;
#pragma unroll
  for (int i = 0; i < L::kDma; ++i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(k0, (lds_void*)(kbuf + 1024 * i), 16, k_src[i], 0,
                                             0, kPolicy);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(k1, (lds_void*)(kbuf + L::kPageBytes + 1024 * i),
                                             16, k_src[i], 0, 0, kPolicy);
  }
#pragma unroll
  for (int i = 0; i < DecodeRegs<D>::kLoads; ++i) {
    r.v[0][i] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(v0, v_off + 1024 * i, 0, kPolicy));
    r.v[1][i] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(v1, v_off + 1024 * i, 0, kPolicy));
  }
}

// Transposed read of 4 key rows x 16 head-dim entries of a V page (ds_read_b64_tr_b16).
__device__ __forceinline__ uint2 read_tr(const uint8_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  return __builtin_bit_cast(uint2, v);
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
// a.k_new / a.v_new into its pool slot, and waits for the stores before it issues the
// loads of the step that holds the slot.  No other split reads that slot, so the result
// equals appending first and then decoding.
// Partials of plain decode travel between CUs, possibly on different XCDs, whose L2s are
// not kept coherent for ordinary accesses.  They are therefore stored and loaded with
// device-scope cache policy (SC1: the store writes through to the device's coherence
// point, the load does not take a possibly stale cached line), which makes the heavy
// cache write-back and invalidate of a device-scope fence unnecessary: a wave waits for
// its partial stores to complete before it counts its arrival, and the merging wave
// loads the partials only after its count returned.
constexpr int kDeviceScope = 16;  // buffer cache policy bit SC1

__device__ __forceinline__ void store_f32x4_device(float* base, uint32_t bytes, uint32_t off,
                                                   f32x4 v) {
  const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(base, 0, bytes, 0x00020000);
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rsrc, off, 0, kDeviceScope);
}

// Merge of the n >= 2 split partials of the G query heads of one (task, kv head), by one
// wave: lanes 8j .. 8j + 7 take head j (a second pass takes heads 8 .. 15), each lane D/8
// consecutive head-dim entries.  With M = max_s m_s and w_s = 2^(m_s - M), the row is
// sum_s w_s o_s / sum_s w_s l_s and its LSE ln(sum_s w_s l_exact_s) + M ln 2.  Every sum
// runs over the splits in split order, so the result does not depend on which split
// finished last.
template <int D>
__device__ __forceinline__ void merge_kv_head(const DecodeArgs& a, int task, int kv_h, int n) {
  constexpr int kPer = D / 8;  // head-dim entries per lane
  constexpr int kBatch = 4;    // splits whose partials are loaded together
  const int lane = threadIdx.x & 63;
  const int hh = lane >> 3, sub = lane & 7;
  const int G = a.group;
  // one buffer over the group's partial rows (wave-uniform); a lane's row is its offset
  const int64_t row0 = (int64_t)task * a.num_q_heads + kv_h * G;
  const auto ml = __builtin_amdgcn_make_buffer_rsrc(a.part_ml + row0 * a.max_splits * 4, 0,
                                                    G * a.max_splits * 16, 0x00020000);
  const auto po = __builtin_amdgcn_make_buffer_rsrc(a.part_o + row0 * a.max_splits * D, 0,
                                                    G * a.max_splits * D * 4, 0x00020000);
  for (int j0 = 0; j0 < G; j0 += 8) {
    const int j = j0 + hh;
    const bool ok = j < G;
    const int64_t row = row0 + (ok ? j : 0);
    const int rs = (ok ? j : 0) * a.max_splits;  // the lane's first partial row
    float mx = kNoMax;
    for (int s0 = 0; s0 < n; s0 += 16) {
      float m[16];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        m[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             ml, 16 * (rs + min(s0 + i, n - 1)), 0, kDeviceScope));
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, m[i]);  // repeats of split n-1 are harmless
    }
    f32x4 acc[kPer / 4];
#pragma unroll
    for (int k = 0; k < kPer / 4; ++k) acc[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    float l_round = 0.0f, l_ex = 0.0f;
    for (int s0 = 0; s0 < n; s0 += kBatch) {
      f32x4 st[kBatch], src[kBatch][kPer / 4];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int sp = min(s0 + i, n - 1);  // past n: a valid slot, not summed below
        st[i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                              ml, 16 * (rs + sp), 0, kDeviceScope));
#pragma unroll
        for (int k = 0; k < kPer / 4; ++k)
          src[i][k] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                    po, 4 * ((rs + sp) * D + kPer * sub + 4 * k), 0,
                                                    kDeviceScope));
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        if (s0 + i < n) {
          const float w = fast_exp2(st[i][0] - mx);
          l_round += w * st[i][1];
          l_ex += w * st[i][2];
#pragma unroll
          for (int k = 0; k < kPer / 4; ++k) acc[k] += w * src[i][k];
        }
      }
    }
    if (ok) {
      const float inv = 1.0f / l_round;
      uint16_t* orow = a.out + row * D + kPer * sub;
#pragma unroll
      for (int k = 0; k < kPer / 8; ++k) {
        const u32x4 w = {pack_bf16x2(acc[2 * k][0] * inv, acc[2 * k][1] * inv),
                         pack_bf16x2(acc[2 * k][2] * inv, acc[2 * k][3] * inv),
                         pack_bf16x2(acc[2 * k + 1][0] * inv, acc[2 * k + 1][1] * inv),
                         pack_bf16x2(acc[2 * k + 1][2] * inv, acc[2 * k + 1][3] * inv)};
        store_u32x4(orow + 8 * k, w);
      }
      if (a.lse && sub == 0) a.lse[row] = (mx + __log2f(l_ex)) * kLn2;
    }
  }
}

template <int D, bool kShared, bool kAppend, int kWaves>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_split_kernel(DecodeArgs a) {
  const int lane = threadIdx.x & 63;
  // the wave index is uniform across the wave: say so, so the item and every address
  // derived from it stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int item_id = blockIdx.x * kWaves + wave;
  // K pages of the two steps in flight, one region per wave (2 pages per step)
  using L = KLds<D>;
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[kWaves * 2 * L::kPageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds1[kWaves * 2 * L::kPageBytes];
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

  uint32_t k_src[L::kDma];
#pragma unroll
  for (int i = 0; i < L::kDma; ++i) k_src[i] = L::src_offset(i, lane);
  // S^T operand c of a page: row `col`, granule 4c + grp; granules 4c + grp for even and
  // odd c differ only in bit 2 and in g / 8 = c / 2, which adds 1 KB
  const uint32_t k_rd_even = L::lds_offset(col, grp), k_rd_odd = L::lds_offset(col, 4 + grp);
  const uint32_t v_off = (uint32_t)(16 * lane);  // this lane's 16 bytes of each 1 KB V load
  // LDS byte offsets: where this lane's V granules go (load i of a page covers rows
  // i * rpl + lane / kNG), and the transposed operand reads of head-dim tile t: rows
  // 4 grp + gl / 4, entries 16t + 4 (gl % 4) .. + 3 for lane gl of 16-lane group grp,
  // so lane l receives V[4 grp + e][16t + l % 16] in slot e.
  using VL = VLds<D>;
  constexpr int kRpl = 1024 / (2 * D);  // rows per 1 KB load
  uint32_t v_wr[DecodeRegs<D>::kLoads];
#pragma unroll
  for (int i = 0; i < DecodeRegs<D>::kLoads; ++i)
    v_wr[i] = VL::offset(i * kRpl + lane / VL::kNG, lane % VL::kNG);
  const int gl = lane & 15, vr = 4 * grp + (gl >> 2);
  uint32_t v_rd[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t)
    v_rd[t] = (uint32_t)(vr * 2 * D + 32 * (t ^ VL::vsw(vr)) + 8 * (gl & 3));

  // Page ids come from scalar loads, so that no wait for one ever waits for the K/V
  // loads in flight.  A page past the context (or with an invalid id) gets a buffer
  // descriptor of range 0: its loads return zeros without touching memory, and the
  // masks below keep those slots out of the result.  An invalid id is reported once, at
  // the end.
  bool flag_error = false;
  auto page_ref = [&](int lp, int64_t& blk) -> int {
    const bool in = lp < npages;
    const int32_t p = load_page_id(bt_row, in ? lp : npages - 1);
    const bool bad = p < 0 || p >= a.num_pages;
    if (bad && in) flag_error = true;
    const bool use = in && !bad;
    blk = ((int64_t)(use ? p : 0) * a.num_kv_heads + kv_h) * kBlk;
    return use ? (int)kBlk : 0;
  };
  // the split that appends the newest token (kAppend)
  const bool appender = kAppend && kend == kv_len;
  auto load = [&](DecodeRegs<D>& r, uint8_t* kbuf, int k, auto policy_tag) {
    if (kAppend && appender && k + kDecodeStep >= kv_len) {
      // this step holds the appended slot: its stores must have completed first
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) expcnt(0) lgkmcnt(0)
      __atomic_signal_fence(__ATOMIC_SEQ_CST);  // and no load is moved above the wait
    }
    int64_t b0, b1;
    const int n0 = page_ref(k / kPage, b0), n1 = page_ref(k / kPage + 1, b1);
    load_step<D, decltype(policy_tag)::value>(
        r, kbuf, block_rsrc(kpool + b0, n0), block_rsrc(kpool + b1, n1),
        block_rsrc(vpool + b0, n0), block_rsrc(vpool + b1, n1), k_src, v_off);
  };

  f32x4 o[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t) o[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;

  // tail_tag: whether this step may hold keys at or past kend.  Only a split's last step
  // can (every earlier step ends at or below kend), so the others skip the masks.
  auto compute = [&](DecodeRegs<D>& cur, const uint8_t* kbuf, int k, auto tail_tag) {
    // S^T for page t: s[t][e] is key k + 16*t + 4*grp + e of query head `col`
    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < D / 32; ++c) {
        const uint32_t off = t * L::kPageBytes + 1024 * (c >> 1) + ((c & 1) ? k_rd_odd : k_rd_even);
        const u32x4 kk = *reinterpret_cast<const u32x4*>(kbuf + off);
        s[t] = mfma16(as_bf16x8(kk), qf[c], s[t]);
      }
    }
    // keys at or past kend (the context's end, or the shared prefix's) are not this item's
    const bool tail = decltype(tail_tag)::value && k + 2 * kPage > kend;
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
    // V over the K copy (its reads are done: the MFMAs above consumed them), then the
    // transposed operands back; LDS keeps one wave's accesses in order
    uint8_t* vbuf = const_cast<uint8_t*>(kbuf);
#pragma unroll
    for (int hp = 0; hp < 2; ++hp)
#pragma unroll
      for (int i = 0; i < DecodeRegs<D>::kLoads; ++i)
        *reinterpret_cast<u32x4*>(vbuf + hp * L::kPageBytes + v_wr[i]) = cur.v[hp][i];
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
      uint2 v0 = read_tr(vbuf + v_rd[t]);
      uint2 v1 = read_tr(vbuf + L::kPageBytes + v_rd[t]);
      if (tail) {  // V slots past kend must not reach the MFMA (NaN * 0 = NaN)
        v0 = keep_first4(v0, kend - (k + 4 * grp));
        v1 = keep_first4(v1, kend - (k + 16 + 4 * grp));
      }
      const u32x4 vv = {v0.x, v0.y, v1.x, v1.y};
      o[t] = mfma16(as_bf16x8(vv), pb, o[t]);
    }
  };

  if constexpr (kAppend) {
    // The split that ends the context appends its newest token before reading: the K
    // and V rows of slot pos % 16.  Its loads of earlier steps overlap the stores;
    // the step that holds the slot waits for them (in `load`), so its loads return the
    // new token.  No other wave reads this page (splits end on 32-key boundaries, other
    // kv heads' blocks are whole 4 KB pages, and pages past a context are never read),
    // and this wave's earlier steps read earlier pages, so no load in this kernel can
    // have put a stale copy of the slot in this CU's L1.
    if (appender) {
      const int pos = kv_len - 1, slot = pos % kPage;
      const int32_t p = bt_row[pos / kPage];
      if (p >= 0 && p < a.num_pages) {
        const int64_t row = (int64_t)td.row_start * a.num_kv_heads + kv_h;
        const int64_t blk = ((int64_t)p * a.num_kv_heads + kv_h) * (int64_t)(kPage * D);
        uint16_t* kdst = const_cast<uint16_t*>(a.k_pool) + blk + (int64_t)slot * D;
        uint16_t* vdst = const_cast<uint16_t*>(a.v_pool) + blk + (int64_t)slot * D;
        const uint16_t* kn = a.k_new + row * D;
        const uint16_t* vn = a.v_new + row * D;
        if (lane < D / 8) {
          store_u32x4(kdst + 8 * lane, load_u32x4(kn + 8 * lane));
          store_u32x4(vdst + 8 * lane, load_u32x4(vn + 8 * lane));
        }
      } else {
        flag_error = true;
      }
    }
  }

  // Two buffers in ping-pong: the next step is in flight while one is used.  Every load
  // is issued on straight-line code (the last one or two steps are peeled off the
  // loop), so the same loads are outstanding on every path into a compute and its wait
  // leaves the next step in flight.
  auto stream = [&](auto policy_tag) {
    DecodeRegs<D> ra, rb;
    uint8_t* ka = k_lds0 + wave * 2 * L::kPageBytes;
    uint8_t* kb = k_lds1 + wave * 2 * L::kPageBytes;
    const int nsteps = (kend - kbeg + kDecodeStep - 1) / kDecodeStep;
    if (nsteps <= 0) return;
    // the scheduling barriers keep each step's loads issued before the reads of the
    // step before it (which would otherwise be hoisted above them, and wait with the
    // next step not yet in flight)
    const std::false_type inner;
    const std::true_type last;
    load(ra, ka, kbeg, policy_tag);
    int k = kbeg;
    for (int i = 0; i + 2 < nsteps; i += 2, k += 2 * kDecodeStep) {
      load(rb, kb, k + kDecodeStep, policy_tag);
      __builtin_amdgcn_sched_barrier(0);
      compute(ra, ka, k, inner);
      load(ra, ka, k + 2 * kDecodeStep, policy_tag);
      __builtin_amdgcn_sched_barrier(0);
      compute(rb, kb, k + kDecodeStep, inner);
    }
    if (k + kDecodeStep < kend) {
      load(rb, kb, k + kDecodeStep, policy_tag);
      __builtin_amdgcn_sched_barrier(0);
      compute(ra, ka, k, inner);
      compute(rb, kb, k + kDecodeStep, last);
    } else {
      compute(ra, ka, k, last);
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
  if constexpr (!kShared) {
    const int nsplit = td.aux;
    if (nsplit == 1) {
      // the task's only split: its rows are final (the merge of one partial is this
      // same arithmetic: weight 2^0 = 1, output o / l)
      if (col_ok) {
        const float inv = 1.0f / l_tot;
        uint16_t* orow = a.out + qrow * D;
#pragma unroll
        for (int t = 0; t < D / 16; ++t) {
          const uint2 w = {pack_bf16x2(o[t][0] * inv, o[t][1] * inv),
                           pack_bf16x2(o[t][2] * inv, o[t][3] * inv)};
          *reinterpret_cast<uint2*>(orow + 16 * t + 4 * grp) = w;
        }
        if (a.lse && grp == 0) a.lse[qrow] = (m_ref + __log2f(l_ex)) * kLn2;
      }
      return;
    }
  }
  if (col_ok) {
    const int64_t slot =
        ((int64_t)ctask * a.num_q_heads + kv_h * G + chead) * a.max_splits + split;
    float* po = a.part_o + slot * D;
    const f32x4 ml = {m_ref, l_tot, l_ex, 0.0f};
    if constexpr (kShared) {  // merged by a second kernel
#pragma unroll
      for (int t = 0; t < D / 16; ++t)
        *reinterpret_cast<f32x4*>(po + 16 * t + 4 * grp) = o[t];
      if (grp == 0) *reinterpret_cast<f32x4*>(a.part_ml + slot * 4) = ml;
    } else if (a.tickets) {  // merged in this kernel, possibly by a wave on another XCD
      // One buffer over the partial rows of this (task, kv head), the same for the whole
      // wave, and each lane's row as its offset: a per-lane buffer base would make the
      // compiler loop over the distinct bases around every store.
      const int64_t row0 = ((int64_t)ctask * a.num_q_heads + kv_h * G) * a.max_splits;
      const uint32_t r = (uint32_t)(chead * a.max_splits + split);
      const uint32_t nrows = (uint32_t)(G * a.max_splits);
#pragma unroll
      for (int t = 0; t < D / 16; ++t)
        store_f32x4_device(a.part_o + row0 * D, nrows * D * 4, 4 * (r * D + 16 * t + 4 * grp), o[t]);
      if (grp == 0) store_f32x4_device(a.part_ml + row0 * 4, nrows * 16, 16 * r, ml);
    } else {  // merged by the merge kernel
#pragma unroll
      for (int t = 0; t < D / 16; ++t)
        *reinterpret_cast<f32x4*>(po + 16 * t + 4 * grp) = o[t];
      if (grp == 0) *reinterpret_cast<f32x4*>(a.part_ml + slot * 4) = ml;
    }
  }
  if constexpr (!kShared) {
    if (a.tickets) {
      // Arrival count of this (task, kv head); the split that completes it merges.  The
      // partial stores complete before the count is taken, and the merge's loads issue
      // only after it returned (both device-scope, see store_f32x4_device).
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      int arrived = 0;
      if (lane == 0)
        arrived = __hip_atomic_fetch_add(a.tickets + (int64_t)first_task * a.num_kv_heads + kv_h,
                                         1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      arrived = __shfl(arrived, 0, 64);
      asm volatile("" ::: "memory");
      if (arrived != td.aux - 1) return;
      merge_kv_head<D>(a, first_task, kv_h, td.aux);
    }
  }
}

// One wave per (task, query head): combine the task's split partials.  kSkipSingle: a
// task with one split already wrote its rows (plain decode).
template <int D, bool kSkipSingle>
__global__ __launch_bounds__(kMergeWaves * 64) void decode_merge_kernel(DecodeArgs a) {
  // wave-uniform and 32-bit (the launch has num_tasks * Hq < 2^31 waves)
  const int row = (int)blockIdx.x * kMergeWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= a.num_tasks * a.num_q_heads) return;
  const int task = row / a.num_q_heads;
  const int n = a.tasks[task].aux;
  if (kSkipSingle && n == 1) return;
  const int64_t r = row;
  merge_partials<D>(a.part_ml + r * a.max_splits * 4, 4, a.part_o + r * a.max_splits * D, D,
                    n, a.out + r * D, a.lse ? a.lse + r : nullptr);
}

template <int D, bool kShared, bool kAppend>
hipError_t launch(const DecodeArgs& a, hipStream_t stream) {
  if (a.num_items > 0) {
    if (decode_waves(a.num_items) == kBigWaves) {
      const int blocks = (a.num_items + kBigWaves - 1) / kBigWaves;
      hipLaunchKernelGGL((decode_split_kernel<D, kShared, kAppend, kBigWaves>), dim3(blocks),
                         dim3(kBigWaves * 64), 0, stream, a);
    } else {
      const int blocks = (a.num_items + kSmallWaves - 1) / kSmallWaves;
      hipLaunchKernelGGL((decode_split_kernel<D, kShared, kAppend, kSmallWaves>), dim3(blocks),
                         dim3(kSmallWaves * 64), 0, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (!kShared && a.tickets) return hipSuccess;  // merged inside the split kernel
  const int64_t rows = (int64_t)a.num_tasks * a.num_q_heads;
  if (rows >= INT32_MAX - kMergeWaves) return hipErrorInvalidValue;
  if (rows > 0) {
    const int blocks = (int)((rows + kMergeWaves - 1) / kMergeWaves);
    hipLaunchKernelGGL((decode_merge_kernel<D, !kShared>), dim3(blocks), dim3(kMergeWaves * 64),
                       0, stream, a);
  }
  return hipGetLastError();
}

// Every variant of each head size is instantiated explicitly: the host pass otherwise
// emits the launch stub of only one of two specialisations that differ in a bool.
template __global__ void decode_split_kernel<128, false, false, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<128, false, false, kSmallWaves>(DecodeArgs);
template __global__ void decode_split_kernel<128, true, false, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<128, true, false, kSmallWaves>(DecodeArgs);
template __global__ void decode_split_kernel<128, false, true, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<128, false, true, kSmallWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, false, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, false, kSmallWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, true, false, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, true, false, kSmallWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, true, kBigWaves>(DecodeArgs);
template __global__ void decode_split_kernel<64, false, true, kSmallWaves>(DecodeArgs);

}  // namespace kern

int decode_waves(int32_t num_items) {
  return num_items >= kern::kBigLaunchItems ? kern::kBigWaves : kern::kSmallWaves;
}

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
