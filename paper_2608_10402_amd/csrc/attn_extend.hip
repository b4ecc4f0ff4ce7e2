// Extend attention over the paged KV pool (and full prefill, which is the same kernel
// with prefix 0): the compute of a resumed task that kept its cache (TideRL,
// Continuous Task Batching, Sections 4 and 4.2) and of the recompute that an evicted
// cache forces (challenge C1, Section 2.2).
//
// Method: FlashAttention-2-style streaming softmax (Dao 2023; online softmax of Milakov
// & Gimelshein 2018) over K/V gathered page by page (PagedAttention, Kwon et al. 2023),
// laid out for CDNA4:
//   * A workgroup of 8 waves owns one (task, kv head, block of tokens) item.  Its 256
//     query rows are the (token, head) pairs of the block for every query head of the kv
//     head, so each K/V tile in LDS serves all G grouped heads at once.  One workgroup
//     fills a CU: two waves per SIMD.
//   * Two waves per SIMD (waves w and w+4) share the SIMD in a fixed rotation.  Every
//     wave alternates a matrix phase (P.V of the previous tile, then S = K.Q^T of the
//     current one: 32 MFMAs) and vector work (mask, running max, exp2, bf16 packing,
//     row sums).  Workgroup barriers cut each tile into three slots: in the first two,
//     one group's MFMAs overlap the other group's VALU work; in the third, no MFMA runs
//     and both groups evaluate their exponentials, because v_exp_f32 does not overlap
//     MFMAs on the same SIMD.
//   * K/V tiles of 64 keys (4 pages) go from HBM straight into LDS with buffer loads
//     that write LDS (no staging registers).  Four LDS buffers: in its vector phase of
//     tile i every wave streams one page of tile i+3 (waves 0-3 the K pages, waves 4-7
//     the V^T pages), so a tile has about four phases to arrive.  Page ids are read
//     with scalar loads.
//   * S^T = K.Q^T per wave with v_mfma_f32_32x32x16_bf16: keys are the MFMA rows,
//     queries the columns, so every lane owns one query row and its softmax statistics
//     need one exchange between lanes l and l^32 (v_permlane32_swap, a VALU op).
//   * Key rows are read in the perm32 order, which leaves each lane holding runs of 8
//     consecutive keys: the probabilities convert straight into the B operand of the
//     O^T += V^T.P^T MFMA with no shuffle.  V pages are stored transposed in the pool
//     (head-dim major, 16 token slots contiguous), so V^T operands are plain 16-byte LDS
//     reads.  K rows are XOR-swizzled by 16-byte granule in LDS so that the 64 lanes of an
//     operand read hit distinct banks; V^T rows swap their 16-byte halves every 8 rows.
//   * Scores stay raw until one FMA applies sm_scale*log2(e) and subtracts the running
//     max before v_exp_f32.  The running max is only raised when a tile exceeds it by
//     more than kRescaleSlack, so the O rescale is skipped on almost every tile.
//   * Causal masking is applied only on tiles that cross the diagonal.  On the last
//     tile, V operands of key slots at or beyond the task's length are zeroed in
//     registers, so NaN/Inf garbage in unused pool slots can never reach the output.
#include <type_traits>

#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWaves = 8;  // two groups of four, one phase apart
constexpr int kThreads = kWaves * 64;

template <int D>
struct ES {
  static constexpr int kNG = D / 8;             // 16-byte granules per K row
  static constexpr int kRB = 16 / kNG;          // K rows per 256-byte LDS bank row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kPageBytes = kPage * kRowBytes;
  static constexpr int kTileBytes = 4 * kPageBytes;  // 64 keys
  static constexpr int kDma = kPageBytes / 1024;     // 1 KB wave transfers per page
  static constexpr int kRowsPerDma = 1024 / kRowBytes;
  static constexpr int kLoads = 2 * kDma;            // vector-memory ops per streamed tile
  static_assert(kDma >= 1 && kRowsPerDma * kRowBytes == 1024, "page split");
};

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from `page` (a buffer of `bytes` bytes; reads past it return 0) at
// byte offset `voff`, written by the buffer unit straight into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(const uint8_t* page, int bytes, uint32_t voff, uint8_t* lds) {
  const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(page), 0, bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)lds, 16, voff, 0, 0, 0);
}

// Swizzled position of granule g in K row r.
template <int D>
__device__ __forceinline__ int kswz(int r, int g) {
  return g ^ ((r / ES<D>::kRB) % ES<D>::kNG);
}

// Position (0/1) of 16-byte half `hh` of V^T row d in LDS: rows d and d+8 share banks,
// so the halves of rows with bit 3 set are swapped.
__device__ __forceinline__ int vswz(int d, int hh) { return hh ^ ((d >> 3) & 1); }

// s_waitcnt vmcnt(N) (gfx9 encoding; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier between phases, with no memory fence: LDS tiles are published by
// each wave's own vmcnt wait before it, and outstanding prefetches must stay in flight.
// The scheduling barriers keep every instruction in the phase it was written in (the
// compiler would otherwise move MFMAs, which touch no memory, across s_barrier).
__device__ __forceinline__ void phase_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// Values of lanes l and l^32 side by side.  v_permlane32_swap trades lanes 32-63 of its
// first operand with lanes 0-31 of its second; starting from two copies of v, the first
// ends up holding the low half twice and the second the high half twice.  It is issued
// by hand because the compiler folds the intrinsic's second result into its first.  The
// s_nop provides the wait states this instruction needs after a VALU write of its inputs.
__device__ __forceinline__ void lane_pair(float v, float& x, float& y) {
  uint32_t lo = __builtin_bit_cast(uint32_t, v), hi = lo;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(lo), "+v"(hi));
  x = __builtin_bit_cast(float, lo);
  y = __builtin_bit_cast(float, hi);
}

__device__ __forceinline__ float pair_max(float v) {
  float x, y;
  lane_pair(v, x, y);
  return fmaxf(x, y);
}

__device__ __forceinline__ float pair_sum(float v) {
  float x, y;
  lane_pair(v, x, y);
  return x + y;
}

// kLse: also keep the exact fp32 sum of the probabilities, so the returned log-sum-exp is
// the true one; the output itself is normalised by the sum of the bf16-rounded weights
// that the P.V product used.
// kSplit: the work list is the split-KV plan's.  A workgroup walks the key tiles
// [t_begin, t_end) of its item; a chunk of a split item writes its unnormalised fp32
// output and statistics to the partial buffers for extend_merge_kernel, an unsplit item
// writes its rows as usual.
template <int D, bool kLse, bool kSplit>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void extend_attn_kernel(ExtendArgs a) {
  using S = ES<D>;
  constexpr int kDC = D / 16;  // 16-wide head-dim chunks of QK^T
  constexpr int kDT = D / 32;  // 32-row head-dim tiles of O^T
  // Tile buffers: K at offset 0, V^T at kTileBytes.  One array per buffer lets the
  // compiler track in-flight LDS writes per buffer, so reading one buffer never waits
  // for the prefetch into another.
  __shared__ __attribute__((aligned(1024))) uint8_t kv_lds0[2 * S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kv_lds1[2 * S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kv_lds2[2 * S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kv_lds3[2 * S::kTileBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool v_half = wave >= 4;  // waves 4-7: V^T pages, one phase behind; 0-3: K pages
  const int pw = wave & 3;        // page of every tile this wave fetches
  const int q = lane & 31, h = lane >> 5;

  ExtendItem it;
  int tbase = 0, split = -1, pbase = 0, t_stop = 0;
  if constexpr (kSplit) {
    const ExtendChunkItem ci = a.chunk_items[blockIdx.x];
    it = ExtendItem{ci.task, ci.kv_head, ci.tok0, ci.ntok};
    tbase = ci.t_begin;
    t_stop = ci.t_end;
    split = ci.split;
    pbase = ci.pbase;
  } else {
    it = a.items[blockIdx.x];
  }
  if (it.ntok == 0) return;  // padding slot of the XCD-interleaved work list
  const TaskDesc td = a.tasks[it.task];
  const int P = td.prefix;
  const int seq_len = td.prefix + td.extend;
  const int G = a.group;
  const int npages = (seq_len + kPage - 1) / kPage;
  const int kend = P + it.tok0 + it.ntok;     // keys needed by the last row
  // Tiles walked, counted from tile tbase: below, `tile` is this local index (it picks
  // the LDS buffers) and tbase + tile the key tile (64 keys from key 0).
  const int ntiles = kSplit ? t_stop - tbase : (kend + 63) / 64;
  const int n_full = (P + it.tok0 + 1) / 64;  // tiles every row sees completely

  // ---- K/V streaming: waves 0-3 fetch the K pages, waves 4-7 the V^T pages ---------
  const int32_t* bt = a.block_table + (int64_t)it.task * a.bt_stride;
  const uint8_t* src_pool = reinterpret_cast<const uint8_t*>(v_half ? a.v_pool : a.k_pool);
  const int lds_half = v_half ? S::kTileBytes : 0;  // V^T lives after K in each buffer
  uint32_t src_off[S::kDma];  // this lane's byte offset inside a K or V^T page, per transfer
#pragma unroll
  for (int i = 0; i < S::kDma; ++i) {
    const int r = i * S::kRowsPerDma + lane / S::kNG;  // K row inside the page
    const int d = i * 32 + lane / 2;                   // V^T row (head-dim entry)
    src_off[i] = v_half ? (uint32_t)(d * (kPage * 2) + vswz(d, lane & 1) * 16)
                        : (uint32_t)(r * S::kRowBytes + kswz<D>(r, lane % S::kNG) * 16);
  }
  bool bad_page = false;
  // Page id of this wave's page of `tile` (a scalar load), or kPastEnd for a page past
  // the sequence (a value no page id can take).
  constexpr int64_t kPastEnd = -(int64_t(1) << 40);
  auto page_word = [&](int tile) -> int64_t {
    const int lp = (tbase + tile) * 4 + pw;
    return lp < npages ? (int64_t)load_page_id(bt, lp) : kPastEnd;
  };
  // Every step issues the same number of loads on every wave, so the vmcnt waits below
  // hold on every path.  A tile past the item (live == false), a page past the sequence
  // and an invalid page id are read through a zero-length buffer, which returns zeros
  // without touching memory; their keys are masked and their V slots zeroed.
  auto stream_tile = [&](int64_t word, uint8_t* kv, bool live) {
    const bool past = word == kPastEnd;
    const bool bad = live && !past && (word < 0 || word >= a.num_pages);
    bad_page |= bad;
    const bool use = live && !past && !bad;
    const int64_t blk = ((use ? word : 0) * a.num_kv_heads + it.kv_head) *
                        (int64_t)S::kPageBytes;
    const int bytes = use ? S::kPageBytes : 0;
#pragma unroll
    for (int i = 0; i < S::kDma; ++i)
      dma16(src_pool + blk, bytes, src_off[i], kv + lds_half + pw * S::kPageBytes + i * 1024);
  };

  // ---- this lane's query row: (token tk of the block, head j of the group) -----------
  const int r = wave * 32 + q;
  const int tk = r / G, j = r - (r / G) * G;
  const bool row_valid = tk < it.ntok;
  const int lim = row_valid ? P + it.tok0 + tk : -1;  // last visible key position
  const int64_t qrow = (int64_t)(td.row_start + it.tok0 + tk) * a.num_q_heads +
                       it.kv_head * G + j;
  bf16x8 qf[kDC];
#pragma unroll
  for (int cc = 0; cc < kDC; ++cc)
    qf[cc] = as_bf16x8(row_valid ? load_u32x4(a.q + qrow * D + 16 * cc + 8 * h) : zero_u32x4());

  // ---- prologue: tiles 0..2 in flight, tile 0 landed, then the phase offset ---------
  stream_tile(page_word(0), kv_lds0, true);
  __builtin_amdgcn_sched_barrier(0);  // keep the issue order the waits below count on
  stream_tile(page_word(1), kv_lds1, ntiles > 1);
  __builtin_amdgcn_sched_barrier(0);
  stream_tile(page_word(2), kv_lds2, ntiles > 2);
  int64_t next_word = page_word(3);  // page id of the next tile to stream
  wait_vmem<2 * S::kDma>();          // tile 0 (and the query rows) landed
  phase_barrier();
  if (v_half) phase_barrier();  // waves 4-7 start one phase behind

  // per-lane LDS byte offsets of the MFMA operands
  const int krow = perm32(q);
  int k_rd[kDC];
#pragma unroll
  for (int cc = 0; cc < kDC; ++cc) k_rd[cc] = krow * S::kRowBytes + kswz<D>(krow, 2 * cc + h) * 16;
  const int v_rd = krow * (kPage * 2) + vswz(krow, h) * 16;
  const float csc = a.scale_log2;

  f32x16 o[kDT];
#pragma unroll
  for (int t = 0; t < kDT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;
  f32x16 s[2];
  u32x4 pb[4];  // bf16 probabilities of the last softmaxed tile, one 16-key chunk each

  // O^T += V^T.P^T for key tile `tile`, V^T in vb.  With kTail, the V slots of keys at or
  // beyond seq_len are zeroed in registers (0 * NaN would otherwise poison O); only the
  // last tile a workgroup walks can hold such keys.
  auto pv = [&](const uint8_t* vb, int tile, auto tail_tag) {
    constexpr bool kTail = decltype(tail_tag)::value;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      u32x4 msk = {~0u, ~0u, ~0u, ~0u};
      if (kTail) {
        const int nv = seq_len - (tile * 64 + 16 * c + 8 * h);  // valid keys of this lane's 8
#pragma unroll
        for (int w = 0; w < 4; ++w)
          msk[w] = (2 * w < nv ? 0x0000FFFFu : 0u) | (2 * w + 1 < nv ? 0xFFFF0000u : 0u);
      }
      const uint8_t* vp = vb + c * S::kPageBytes + v_rd;
#pragma unroll
      for (int t = 0; t < kDT; ++t) {
        u32x4 vv = load_u32x4(vp + t * 1024);
        if (kTail) vv &= msk;
        o[t] = mfma32(as_bf16x8(vv), as_bf16x8(pb[c]), o[t]);
      }
    }
  };

  // S^T = K.Q^T for the tile held in kb.
  auto qk = [&](const uint8_t* kb) {
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[st][e] = 0.0f;
#pragma unroll
    for (int cc = 0; cc < kDC; ++cc)
#pragma unroll
      for (int st = 0; st < 2; ++st)
        s[st] = mfma32(as_bf16x8(load_u32x4(kb + st * 32 * S::kRowBytes + k_rd[cc])), qf[cc], s[st]);
  };

  // Keep four operand reads in flight ahead of the MFMAs of a matrix phase with n of
  // each: reads first, then MFMA/read pairs, then the last MFMAs.
  auto pipeline = [](auto n_tag) {
    constexpr int n = decltype(n_tag)::value;
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < n - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };

  // The softmax of a tile, in three parts.  o1: causal mask, running max (and the rare
  // rescale of O), then x = s * scale * log2(e) - max in place.  ex: 2^x in place
  // (v_exp_f32, which does not overlap MFMAs on the same SIMD).  o2: bf16 packing into
  // pb and the row sums.
  auto softmax_o1 = [&](int tile) {
    const int kt = tbase + tile;
    if (kt >= n_full) {  // diagonal / tail tile: hide keys past this row's position
      const int kbase = kt * 64 + 8 * h;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kbase + 32 * st + 16 * (e >> 3) + (e & 7) > lim) s[st][e] = -INFINITY;
    }
    float mt = s[0][0];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) mt = fmaxf(mt, s[st][e]);
    mt = pair_max(mt) * csc;
    if (__any(mt > m_ref + kRescaleSlack)) {
      const float m_new = fmaxf(m_ref, mt);
      const float alpha = fast_exp2(m_ref - m_new);
      l_part *= alpha;
      if (kLse) l_exact *= alpha;
#pragma unroll
      for (int t = 0; t < kDT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
      m_ref = m_new;
    }
    const float negm = -m_ref;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[st][e] = fmaf(s[st][e], csc, negm);
  };
  auto softmax_ex = [&]() {
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[st][e] = fast_exp2(s[st][e]);
  };
  auto softmax_o2 = [&]() {
    float lt[4] = {0.0f, 0.0f, 0.0f, 0.0f}, le = 0.0f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = s[st][8 * m + 2 * e], p1 = s[st][8 * m + 2 * e + 1];
          const uint32_t w = pack_bf16x2(p0, p1);
          pb[2 * st + m][e] = w;
          lt[e] = add_bf16x2(w, lt[e]);
          if (kLse) le += p0 + p1;
        }
    l_part += (lt[0] + lt[1]) + (lt[2] + lt[3]);  // short dot2 chains per tile
    if (kLse) l_exact += le;
  };

  // One tile is a round of three slots, each closed by a workgroup barrier:
  //   slot 1: waves 0-3 matrix phase (P.V of tile-1, S of tile)  | waves 4-7 o2 of tile-1
  //   slot 2: waves 0-3 o1 of tile                              | waves 4-7 matrix phase
  //   slot 3: waves 0-3 ex, o2 of tile                          | waves 4-7 o1, ex of tile
  // Every wave runs the same code; only where its second barrier falls differs.  The
  // exponentials of both groups meet in slot 3, where no MFMA runs, and the rest of the
  // vector work overlaps the other group's MFMAs.  In o1 each wave also streams its page
  // of tile+3 (waves 0-3 K, waves 4-7 V^T) into the buffer tile-1 has released, and at
  // the end of the round waits until only its last two tiles are in flight, so tile+1
  // is in LDS before the next round starts.
  auto step = [&](int tile, uint8_t* kv, uint8_t* kv_prev) {
    if (tile > 0) {
      pv(kv_prev + S::kTileBytes, tbase + tile - 1, std::false_type());
      qk(kv);
      pipeline(std::integral_constant<int, 4 * kDT + 2 * kDC>());
    } else {
      qk(kv);
      pipeline(std::integral_constant<int, 2 * kDC>());
    }
    phase_barrier();
    stream_tile(next_word, kv_prev, tile + 3 < ntiles);
    next_word = page_word(tile + 4);
    softmax_o1(tile);
    if (!v_half) phase_barrier();
    softmax_ex();
    if (v_half) phase_barrier();
    softmax_o2();
    wait_vmem<2 * S::kDma>();
    phase_barrier();
  };

  // Four steps per iteration with no conditions inside, so the compiler's view of the
  // loads in flight matches the schedule; the last 0-3 tiles follow the loop.
  int tile = 0;
  for (; tile + 4 <= ntiles; tile += 4) {
    step(tile, kv_lds0, kv_lds3);
    step(tile + 1, kv_lds1, kv_lds0);
    step(tile + 2, kv_lds2, kv_lds1);
    step(tile + 3, kv_lds3, kv_lds2);
  }
  if (tile < ntiles) {
    step(tile, kv_lds0, kv_lds3);
    if (tile + 1 < ntiles) {
      step(tile + 1, kv_lds1, kv_lds0);
      if (tile + 2 < ntiles) step(tile + 2, kv_lds2, kv_lds1);
    }
  }
  const int last = tbase + ntiles - 1;
  switch ((ntiles - 1) & 3) {  // P.V of the last tile
    case 0: pv(kv_lds0 + S::kTileBytes, last, std::true_type()); break;
    case 1: pv(kv_lds1 + S::kTileBytes, last, std::true_type()); break;
    case 2: pv(kv_lds2 + S::kTileBytes, last, std::true_type()); break;
    default: pv(kv_lds3 + S::kTileBytes, last, std::true_type()); break;
  }
  if (!v_half) phase_barrier();  // balances the offset barrier of waves 4-7
  wait_vmem<0>();  // no transfer into LDS may outlive the workgroup

  if (bad_page && lane == 0) atomicOr(a.error_flags, 1);
  const float l_tot = pair_sum(l_part);
  if (kSplit && split >= 0) {
    // Lanes l and l^32 hold the same row, so both take this branch or neither.
    const float l_ex = kLse ? pair_sum(l_exact) : 0.0f;
    if (row_valid) {
      const int64_t slot =
          (int64_t)(pbase + split * it.ntok + tk) * a.num_q_heads + it.kv_head * G + j;
      float* po = a.part_o + slot * D;
#pragma unroll
      for (int t = 0; t < kDT; ++t)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const f32x4 w0 = {o[t][8 * half], o[t][8 * half + 1], o[t][8 * half + 2], o[t][8 * half + 3]};
          const f32x4 w1 = {o[t][8 * half + 4], o[t][8 * half + 5], o[t][8 * half + 6],
                            o[t][8 * half + 7]};
          *reinterpret_cast<f32x4*>(po + 32 * t + 16 * half + 8 * h) = w0;
          *reinterpret_cast<f32x4*>(po + 32 * t + 16 * half + 8 * h + 4) = w1;
        }
      if (h == 0) {
        const f32x4 ml = {m_ref, l_tot, l_ex, 0.0f};
        *reinterpret_cast<f32x4*>(a.part_ml + slot * 4) = ml;
      }
    }
    return;
  }
  if (row_valid) {
    const float inv = 1.0f / l_tot;
    uint16_t* orow = a.out + qrow * D;
#pragma unroll
    for (int t = 0; t < kDT; ++t)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = pack_bf16x2(o[t][8 * half + 2 * e] * inv, o[t][8 * half + 2 * e + 1] * inv);
        store_u32x4(orow + 32 * t + 16 * half + 8 * h, w);
      }
    if (kLse) {
      const float l_ex = pair_sum(l_exact);
      if (h == 0) a.lse[qrow] = (m_ref + __log2f(l_ex)) * kLn2;
    }
  }
}

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
    hipLaunchKernelGGL((extend_attn_kernel<D, true, kSplit>), dim3(a.num_items), dim3(kThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((extend_attn_kernel<D, false, kSplit>), dim3(a.num_items), dim3(kThreads), 0,
                       stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch(const ExtendArgs& a, hipStream_t stream) {
  if (!a.chunk_items) return launch_attn<D, false>(a, stream);
  hipError_t e = launch_attn<D, true>(a, stream);
  if (e != hipSuccess || !a.merge_rows) return e;
  const int64_t waves = (int64_t)a.total_rows * a.num_q_heads;
  if (waves >= INT32_MAX - kMergeWaves) return hipErrorInvalidValue;
  const int blocks = (int)((waves + kMergeWaves - 1) / kMergeWaves);
  hipLaunchKernelGGL((extend_merge_kernel<D>), dim3(blocks), dim3(kMergeWaves * 64), 0, stream, a);
  return hipGetLastError();
}

// Every variant is instantiated explicitly: the host pass otherwise emits the launch stub
// of only one of the specialisations that differ in a bool.
template __global__ void extend_attn_kernel<128, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true, true>(ExtendArgs);

}  // namespace kern

hipError_t launch_extend(const ExtendArgs& a, int head_dim, int waves, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (waves != kern::kWaves) return hipErrorInvalidValue;
  if (head_dim == 128) return kern::launch<128>(a, stream);
  if (head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
