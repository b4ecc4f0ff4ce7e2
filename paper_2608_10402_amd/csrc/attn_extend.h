// attn_extend.h -- the extend attention kernel template (instantiated by attn_extend.hip,
// and with the fused KV-append by attn_extend_append.hip).
//
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
//     fills a CU: two waves per SIMD, 32 query rows per wave.
//   * Every wave runs its own software pipeline over 64-key tiles: while it evaluates
//     the softmax of tile i (VALU and v_exp_f32), its MFMA unit computes P.V of tile i-1
//     and S = K.Q^T of tile i+1.  The three are independent, and interleaved instruction
//     by instruction they overlap: on gfx950 a wave's VALU and transcendental
//     instructions issue while its own MFMAs execute.  The second wave on the SIMD fills
//     the gaps.  One workgroup barrier per tile guards the LDS rings.
//   * K and V tiles of 64 keys (4 pages) go from HBM straight into LDS with buffer loads
//     that write LDS (no staging registers): separate K and V rings of four tiles.  Each
//     wave streams 8 key rows of the K tile and of the V tile three tiles ahead; pages
//     past the sequence, tiles past the item and invalid page ids are read through a
//     zero-length buffer, so every wave issues the same loads on every path and the
//     vmcnt waits hold.  Page ids are scalar loads.
//   * S^T = K.Q^T per wave with v_mfma_f32_32x32x16_bf16: keys are the MFMA rows,
//     queries the columns, so every lane owns one query row and its softmax statistics
//     need one exchange between lanes l and l^32 (v_permlane32_swap).
//   * Key rows are read in the perm32 order, which leaves each lane holding runs of 8
//     consecutive keys: the probabilities convert straight into the B operand of the
//     O^T += V^T.P^T MFMA with no shuffle.  V stays in the pool's [key][d] layout; its
//     V^T operands are read with ds_read_b64_tr_b16, which transposes 4 keys x 16
//     head-dim entries across each 16-lane group (lane j of the group receives element
//     j & 3 of the 8 bytes addressed by lane 4e + (j >> 2), in slot e).  K rows are
//     XOR-swizzled by 16-byte granule in LDS and V rows by 64-byte segment, so that the
//     lanes of an operand read hit distinct banks.
//   * Scores stay raw until one FMA applies sm_scale*log2(e) and subtracts the running
//     max before v_exp_f32.  A row's reference max is only raised when a tile exceeds it
//     by more than kRescaleSlack, so the O rescale is skipped on almost every tile.
//   * Causal masking is applied only on tiles that cross the diagonal.  On the last
//     tile, V operands of key slots at or beyond the task's length are zeroed in
//     registers, so NaN/Inf garbage in unused pool slots can never reach the output.
#pragma once

#include <type_traits>
#include <utility>

#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;

template <int D>
struct ES {
  static constexpr int kNG = D / 8;                  // 16-byte granules per key row
  static constexpr int kRB = 16 / kNG;               // key rows per 256-byte bank row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kTileBytes = 64 * kRowBytes;  // 64 keys
  static constexpr int kRowsPerDma = 1024 / kRowBytes;
  // 1 KB wave transfers per tensor per tile and wave: each wave streams 8 key rows
  static constexpr int kDma = kTileBytes / 1024 / kWaves;
  static constexpr int kGroup = 2 * kDma;  // vector-memory ops a wave issues per tile
  static_assert(kDma * kRowsPerDma == 8, "8 key rows per wave");
};

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// 16 bytes per lane from `base` (a buffer of `bytes` bytes; reads past it return 0) at
// byte offset `voff`, written by the buffer unit straight into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(const uint8_t* base, int bytes, uint32_t voff, uint8_t* lds) {
  const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), 0, bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)lds, 16, voff, 0, 0, 0);
}

typedef __attribute__((address_space(1))) void glb_void;

// 16 bytes from src (one address per lane) written straight into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16_lane(const void* src, uint8_t* lds) {
  __builtin_amdgcn_global_load_lds((glb_void*)src, (lds_void*)lds, 16, 0, 0);
}

// Physical position of 16-byte granule g of K tile row r.
template <int D>
__device__ __forceinline__ int kswz(int r, int g) {
  return g ^ ((r / ES<D>::kRB) % ES<D>::kNG);
}

// XOR applied to the 64-byte segment index of V tile row r (4 segments per row at
// d = 128, 2 at d = 64): the 4 rows x 64 bytes that 32 lanes of a transposed read touch
// then fall in distinct banks.
template <int D>
__device__ __forceinline__ int vseg(int r) {
  return D == 128 ? (r & 3) : ((r >> 1) & 1);
}

// s_waitcnt vmcnt(N) (gfx9 encoding; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier with no memory fence: LDS tiles are published by each wave's own
// vmcnt wait before it, and outstanding prefetches must stay in flight.  The scheduling
// barriers keep every instruction on its side of it.
__device__ __forceinline__ void tile_barrier() {
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

// max(a, b, c) as one v_max3_f32.  Written out because the compiler otherwise quiets
// possible signalling NaNs of MFMA results with extra maxima first; the scores reaching
// these are finite or -inf (masked), never NaN.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Transposed read of 4 keys x 16 head-dim entries of a V tile (ds_read_b64_tr_b16).
__device__ __forceinline__ uint2 read_tr(const uint8_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  return __builtin_bit_cast(uint2, v);
}

// Compile-time loops: f(std::integral_constant<int, i>) for i in [B, E).
template <int B, int... Is, class F>
__device__ __forceinline__ void static_for_seq(std::integer_sequence<int, Is...>, F&& f) {
  (f(std::integral_constant<int, B + Is>()), ...);
}
template <int B, int E, class F>
__device__ __forceinline__ void static_for_range(F&& f) {
  if constexpr (E > B) static_for_seq<B>(std::make_integer_sequence<int, E - B>(), f);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_range<0, N>(f);
}

// kLse: also keep the exact fp32 sum of the probabilities, so the returned log-sum-exp is
// the true one; the output itself is normalised by the sum of the bf16-rounded weights
// that the P.V product used.
// kSplit: the work list is the split-KV plan's.  A workgroup walks the key tiles
// [t_begin, t_end) of its item; a chunk of a split item writes its unnormalised fp32
// output and statistics to the partial buffers for extend_merge_kernel, an unsplit item
// writes its rows as usual.
template <int D, bool kLse, bool kSplit, bool kAppend>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void extend_attn_kernel(ExtendArgs a) {
  using S = ES<D>;
  constexpr int kDC = D / 16;  // 16-wide head-dim chunks of QK^T
  constexpr int kDT = D / 32;  // 32-row head-dim tiles of O^T
  // One array per ring slot, so the compiler tracks in-flight LDS writes per slot and a
  // read of one slot never waits for the prefetch into another.
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds1[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds2[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds3[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds0[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds1[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds2[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds3[S::kTileBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  const int kend = P + it.tok0 + it.ntok;  // keys needed by the last row
  // Tiles walked, counted from tile tbase: below, `i` is this local index and tbase + i
  // the key tile (64 keys from key 0).
  const int ntiles = kSplit ? t_stop - tbase : (kend + 63) / 64;
  const int n_full = (P + it.tok0 + 1) / 64;  // tiles every row sees completely

  // ---- K/V streaming: wave w streams key rows 8w .. 8w+7 of every K and V tile -------
  const int32_t* bt = a.block_table + (int64_t)it.task * a.bt_stride;
  const uint8_t* kpool = reinterpret_cast<const uint8_t*>(a.k_pool);
  const uint8_t* vpool = reinterpret_cast<const uint8_t*>(a.v_pool);
  const int pw = wave >> 1;  // page of the tile these rows sit in
  // a page of one kv head is kPage * kRowBytes bytes; a pool page holds num_kv_heads of them
  const uint32_t page_bytes = (uint32_t)a.num_kv_heads * (kPage * S::kRowBytes);
  const uint8_t* kpool_h = kpool + (int64_t)it.kv_head * (kPage * S::kRowBytes);
  const uint8_t* vpool_h = vpool + (int64_t)it.kv_head * (kPage * S::kRowBytes);
  uint32_t k_src[S::kDma], v_src[S::kDma];  // this lane's byte offsets inside the page block
#pragma unroll
  for (int i = 0; i < S::kDma; ++i) {
    const int r = 8 * wave + i * S::kRowsPerDma + lane / S::kNG;  // tile row
    const int rp = r % kPage;                                       // row inside its page
    const int p = lane % S::kNG;                                    // physical granule
    k_src[i] = (uint32_t)(rp * S::kRowBytes + kswz<D>(r, p) * 16);
    v_src[i] = (uint32_t)(rp * S::kRowBytes + (p ^ (vseg<D>(r) << 2)) * 16);
  }
  const int lds_row0 = 8 * wave * S::kRowBytes;  // where those rows land in a tile
  bool bad_page = false;  // an invalid page id met by a lane of the fused append's pool writes
  uint32_t bad_tile = 0;  // the same for whole-wave page loads, kept in scalar registers
  // This wave's page of local tile t: whether it is live (inside the item and the
  // sequence) and its page id (a scalar load; ids are checked as 32-bit unsigned scalars,
  // so a negative id compares as too large).  Local tiles t < t_live are live (page
  // 4 * (tbase + t) + pw < npages); kNone never is.  The load is unconditional, of entry 0
  // for a page that is not live (every sequence has at least one page), at a 32-bit byte
  // offset from the row that the scalar load takes in its offset register: no branch,
  // no 64-bit address arithmetic, and it can be issued well before the id is used.
  const int t_live = min(ntiles, max(0, (npages - pw - 4 * tbase + 3) / 4));
  const uint32_t pw_off = 4u * (uint32_t)(4 * tbase + pw);
  struct PageRef {
    bool live;
    uint32_t word;
  };
  auto page_ref = [&](int t) -> PageRef {
    const bool live = t < t_live;
    const uint32_t off = live ? 16u * (uint32_t)t + pw_off : 0u;
    return PageRef{live, (uint32_t)*(const_i32*)(reinterpret_cast<const uint8_t*>(bt) + off)};
  };
  // Streams this wave's rows of K tile tk into kbuf and of V tile tv into vbuf (either
  // may be kNone, a load of nothing).  A page past the sequence, a tile past the item and an
  // invalid page id are read through a zero-length buffer: zeros, no memory access.
  // With a fused append (a.k_new), a tile that holds keys at or past the prefix P takes
  // each lane's row from its source: the pool page for keys below P, the new rows for
  // keys P .. seq_len - 1 (which the pool does not hold yet), and for keys past the
  // sequence any valid row (masked out later).  One per-lane-address load per 1 KB, as
  // many as the page path, so the wait counts stay the same.
  constexpr bool fused = kAppend;
  constexpr int kNone = 1 << 30;  // tile index of a load of nothing
  const int64_t new_row0 = (int64_t)td.row_start * a.num_kv_heads + it.kv_head;  // row P, this head
  const uint32_t new_stride_b = (uint32_t)a.num_kv_heads * S::kRowBytes;  // bytes per token row
  auto one_fused = [&](int t, PageRef pg, const uint8_t* pool, const uint16_t* rows,
                       bool is_v, uint8_t* buf) {
    const bool past = !pg.live;
    const bool bad = !past && pg.word >= (uint32_t)a.num_pages;
    const int64_t word = pg.word;
    bad_tile |= (uint32_t)bad;
    const int64_t blk = ((past || bad ? 0 : word) * a.num_kv_heads + it.kv_head) *
                        (int64_t)(kPage * S::kRowBytes);
    // Each lane's address is a wave-uniform base (the new rows of this kv head, or the
    // pool page) plus a 32-bit lane offset.  The offset passes through an empty asm so
    // that the compiler cannot hoist per-lane 64-bit addresses out of the walk: kept live
    // across it they were spilled, and every reload drained the prefetch queue.
    const uint8_t* new_base = reinterpret_cast<const uint8_t*>(rows + new_row0 * D);
    const uint8_t* page_base = pool + blk;
    int ln = lane;  // lane constants too are recomputed here rather than kept live
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int i = 0; i < S::kDma; ++i) {
      const int r = 8 * wave + i * S::kRowsPerDma + ln / S::kNG;  // tile row
      const int p = ln % S::kNG;
      const int g = is_v ? (p ^ (vseg<D>(r) << 2)) : kswz<D>(r, p);  // logical granule
      const int key = (tbase + t) * 64 + r;
      const bool is_new = key >= P && key < seq_len;
      const bool is_old = key < P && !past && !bad;
      // both offsets computed and masked (is_new and is_old exclude each other), so the
      // choice is a select rather than a divergent branch
      const uint32_t off_new = (uint32_t)(key - P) * new_stride_b + 16u * g;
      const uint32_t off_old = (uint32_t)((r % kPage) * S::kRowBytes + 16 * g);
      uint32_t off = (off_new & (0u - (uint32_t)is_new)) | (off_old & (0u - (uint32_t)is_old));
      asm volatile("" : "+v"(off));
      dma16_lane((is_old ? page_base : new_base) + off, buf + lds_row0 + i * 1024);
    }
  };
  // A tile whose keys all lie at or past P (and below seq_len, or zero-filled past it) is
  // streamed from the caller's new rows with the same buffer loads as a pool page: the
  // buffer starts at the tile's first key's row of this kv head, rows are
  // num_kv_heads * D * 2 bytes apart, and lane offsets are constants like the page path's.
  const int64_t new_stride = (int64_t)a.num_kv_heads * S::kRowBytes;  // bytes per token row
  auto one_new = [&](int t, const uint16_t* rows, bool is_v, uint8_t* buf) {
    const int t0 = (tbase + t) * 64;             // first key of the tile, >= P
    const int n = min(seq_len - t0, 64);         // its rows among the new rows (>= 1)
    const uint8_t* base =
        reinterpret_cast<const uint8_t*>(rows + (new_row0 + (int64_t)(t0 - P) * a.num_kv_heads) * D);
    const int bytes = (int)((n - 1) * new_stride) + S::kRowBytes;  // rows past n read as 0
#pragma unroll
    for (int i = 0; i < S::kDma; ++i) {
      const int r = 8 * wave + i * S::kRowsPerDma + lane / S::kNG;  // tile row
      const int p = lane % S::kNG;
      const int g = is_v ? (p ^ (vseg<D>(r) << 2)) : kswz<D>(r, p);  // logical granule
      dma16(base, bytes, (uint32_t)(r * (int)new_stride + g * 16), buf + lds_row0 + i * 1024);
    }
  };
  // The V tile's loads go first: a wait can then cover a group's V tile without its K tile.
  // tk / tv: the local tiles loaded (only used by the fused path).  With fuse_tag false the
  // caller guarantees that both tiles lie below the prefix, and no fused code is emitted.
  // kpg / vpg: the pages of tk and tv, from page_ref.
  auto stream_pages = [&](uint8_t* kbuf, uint8_t* vbuf, int tk, int tv, PageRef kpg, PageRef vpg,
                          auto fuse_tag) {
    constexpr bool kFuse = kAppend && decltype(fuse_tag)::value;
    // pool_h: the pool's block of this kv head in page 0; pages are page_bytes apart
    auto one = [&](PageRef pg, const uint8_t* pool_h, const uint32_t(&src)[S::kDma], uint8_t* buf) {
      const bool ok = pg.word < (uint32_t)a.num_pages;
      bad_tile |= (uint32_t)(pg.live && !ok);
      const bool use = pg.live && ok;
      const uint8_t* base = pool_h + (uint64_t)(use ? pg.word : 0u) * page_bytes;
      const int bytes = use ? kPage * S::kRowBytes : 0;
#pragma unroll
      for (int i = 0; i < S::kDma; ++i) dma16(base, bytes, src[i], buf + lds_row0 + i * 1024);
    };
    // a tile past the item keeps the zero-length path (its keys are never used); a tile
    // wholly at or past P reads the new rows, the one holding key P mixes both sources
    if (kFuse && tv < ntiles && (tbase + tv + 1) * 64 > P) {
      if ((tbase + tv) * 64 >= P) one_new(tv, a.v_new, true, vbuf);
      else one_fused(tv, vpg, vpool, a.v_new, true, vbuf);
    } else {
      one(vpg, vpool_h, v_src, vbuf);
    }
    if (kFuse && tk < ntiles && (tbase + tk + 1) * 64 > P) {
      if ((tbase + tk) * 64 >= P) one_new(tk, a.k_new, false, kbuf);
      else one_fused(tk, kpg, kpool, a.k_new, false, kbuf);
    } else {
      one(kpg, kpool_h, k_src, kbuf);
    }
  };
  auto stream = [&](uint8_t* kbuf, uint8_t* vbuf, int tk, int tv, auto fuse_tag) {
    stream_pages(kbuf, vbuf, tk, tv, page_ref(tk), page_ref(tv), fuse_tag);
  };
  const std::true_type fuse;  // streams that may cross the prefix (fused variant only)

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

  // ---- prologue: K tiles 0-3 and V tiles 0-1 in flight ------------------------------
  // Every iteration t issues one group of loads, V(t+3) then K(t+5), and at its end waits
  // for V(t+1), from the group issued two iterations earlier (and so for K(t+2) too,
  // issued before it); the barrier after it publishes them.  K tiles thus get three
  // iterations to arrive, V tiles two, and iteration t+1 may read the first operands of
  // its P.V product, in V(t), before that barrier.  The prologue issues the earlier
  // tiles in groups of the same shape (the first two with a V load of nothing), so one
  // wait count serves everywhere.
  stream(k_lds0, v_lds2, 0, kNone, fuse);  // K(0)
  __builtin_amdgcn_sched_barrier(0);               // keep the issue order the waits count on
  stream(k_lds1, v_lds3, 1, kNone, fuse);  // K(1)
  __builtin_amdgcn_sched_barrier(0);
  stream(k_lds2, v_lds0, 2, 0, fuse);  // V(0), K(2)
  __builtin_amdgcn_sched_barrier(0);
  stream(k_lds3, v_lds1, 3, 1, fuse);  // V(1), K(3)
  wait_vmem<3 * S::kGroup>();  // the query rows and K(0) landed
  tile_barrier();

  // per-lane LDS byte offsets of the MFMA operands
  const int krow = perm32(q);
  int k_rd[kDC];
#pragma unroll
  for (int cc = 0; cc < kDC; ++cc) k_rd[cc] = krow * S::kRowBytes + kswz<D>(krow, 2 * cc + h) * 16;
  // V^T operand of head-dim tile t, key chunk c, half ld: rows 16c + 8h + 4ld + gl/4,
  // entries 32t + 16(g & 1) + 4 pi(gl & 3) .. + 3, pi = (0, 2, 1, 3), for lane gl of
  // 16-lane group g: lane l then holds head-dim row 32t + 8h + r in register r < 8 and
  // 32t + 16 + 8h + (r - 8) in r >= 8 of the product, as for K.
  const int gl = lane & 15, grp = lane >> 4;
  const int vrow = 8 * h + (gl >> 2);
  const int vpi = (gl & 3) == 1 ? 2 : (gl & 3) == 2 ? 1 : (gl & 3);
  int v_rd[kDT];
#pragma unroll
  for (int t = 0; t < kDT; ++t)
    v_rd[t] = vrow * S::kRowBytes + 64 * (t ^ vseg<D>(vrow)) + 32 * (grp & 1) + 8 * vpi;
  const float csc = a.scale_log2;

  f32x16 o[kDT];
#pragma unroll
  for (int t = 0; t < kDT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;
  f32x16 sa[2], sb[2];  // S of two consecutive tiles (the one in softmax, the next one)
  u32x4 pa[4], pb[4];   // bf16 probabilities of two consecutive tiles, 16-key chunks

  // S^T = K.Q^T for the K tile in kb, into s (tile 0; later tiles are computed inside
  // the pipeline steps).
  auto qk = [&](const uint8_t* kb, f32x16(&s)[2]) {
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

  // O^T += V^T.P^T for the V tile in vb (key tile kt), used for the last tile.  V slots of
  // keys at or beyond seq_len are zeroed in registers (0 * NaN would otherwise poison O);
  // only the last tile a workgroup walks can hold such keys.
  auto pv_tail = [&](const uint8_t* vb, const u32x4(&p)[4], int kt) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int nv = seq_len - (kt * 64 + 16 * c + 8 * h);  // valid keys of this lane's 8
      u32x4 msk;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        msk[w] = (2 * w < nv ? 0x0000FFFFu : 0u) | (2 * w + 1 < nv ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int t = 0; t < kDT; ++t) {
        const uint8_t* vp = vb + (16 * c) * S::kRowBytes + v_rd[t];
        const uint2 lo = read_tr(vp);
        const uint2 hi = read_tr(vp + 4 * S::kRowBytes);
        u32x4 vv = {lo.x, lo.y, hi.x, hi.y};
        vv &= msk;
        o[t] = mfma32(as_bf16x8(vv), as_bf16x8(p[c]), o[t]);
      }
    }
  };

  auto rescale = [&](float alpha) {
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int t = 0; t < kDT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
    }
  };

  constexpr int kAhead = 3;  // operand reads in flight ahead of the MFMAs

  // ---- one pipeline step, scheduled by hand -------------------------------------------
  // The softmax of tile s into pcur (after the causal mask when kDiag), interleaved with
  // the MFMAs of S(next) = K.Q^T into sn and, with kPV, of O^T += V^T.P^T for the
  // previous tile's probabilities pprev and V tile vb.  MFMA j (j < nm): with kPV, the
  // first nPV are the P.V MFMAs (key chunk c = j / kDT, head-dim tile t = j % kDT), so
  // pprev dies halfway, before the S accumulators come alive; the rest are S MFMAs
  // (head-dim chunk cc = js / 2, key block st = js % 2).  Slot m issues the operand read of
  // MFMA m + kAhead, MFMA m and its
  // share of the softmax's vector instructions; a scheduling barrier closes each slot,
  // so the instructions issue in this order and every MFMA's 32 cycles hide about four
  // vector instructions.  Returns the accumulator rescale factor (1 unless the row's
  // reference max was raised), which the caller applies once the P.V MFMAs are issued.
  //
  // The operand reads of the next step's first kAhead MFMAs (P.V of this step's tile,
  // from vb_next) are issued in this step's last slots, into pre_next, before the barrier
  // that ends the step: the tiles they read were published one barrier earlier.  With
  // kPV the first kAhead operands of this step come from pre, read by the step before.
  auto block = [&](auto pv_tag, auto diag_tag, int kt, f32x16(&s)[2], u32x4(&pcur)[4],
                   const u32x4(&pprev)[4], const uint8_t* vb, const uint8_t* kb,
                   f32x16(&sn)[2], const u32x4(&pre)[kAhead], const uint8_t* vb_next,
                   u32x4(&pre_next)[kAhead]) -> float {
    constexpr bool kPV = decltype(pv_tag)::value;
    constexpr bool kDiag = decltype(diag_tag)::value;
    constexpr int nS = 2 * kDC, nPV = 4 * kDT;
    constexpr int nm = kPV ? nS + nPV : nS;
    constexpr int nMask = kDiag ? 32 : 0;
    constexpr int kPerGroup = kLse ? 14 : 12;  // vector ops per 4 probabilities
    constexpr int kHead = 23;                  // max, exchange, reference update
    constexpr int nOps = nMask + kHead + 8 * kPerGroup + 1;
    const int kbase = kt * 64 + 8 * h;
    const f32x16 zero16 = {};

    u32x4 opnd[nm];
    auto issue = [&](auto j_tag) {
      constexpr int j = decltype(j_tag)::value;
      if constexpr (j >= nm) {  // the next step's P.V MFMA j - nm
        constexpr int c = (j - nm) / kDT, t = (j - nm) % kDT;
        const uint8_t* vp = vb_next + (16 * c) * S::kRowBytes + v_rd[t];
        const uint2 lo = read_tr(vp);
        const uint2 hi = read_tr(vp + 4 * S::kRowBytes);
        pre_next[j - nm] = u32x4{lo.x, lo.y, hi.x, hi.y};
        asm volatile("" ::"v"(lo), "v"(hi));  // issued here, not sunk past the barrier
      } else if constexpr (kPV && j < kAhead) {
        opnd[j] = pre[j];
      } else {
        if constexpr (kPV && j < nPV) {
          constexpr int c = j / kDT, t = j % kDT;
          const uint8_t* vp = vb + (16 * c) * S::kRowBytes + v_rd[t];
          const uint2 lo = read_tr(vp);
          const uint2 hi = read_tr(vp + 4 * S::kRowBytes);
          opnd[j] = u32x4{lo.x, lo.y, hi.x, hi.y};
        } else {
          constexpr int js = kPV ? j - nPV : j;
          constexpr int cc = js / 2, st = js % 2;
          opnd[j] = load_u32x4(kb + st * 32 * S::kRowBytes + k_rd[cc]);
        }
      }
    };
    auto mfma = [&](auto j_tag) {
      constexpr int j = decltype(j_tag)::value;
      if constexpr (kPV && j < nPV) {
        constexpr int c = j / kDT, t = j % kDT;
        o[t] = mfma32(as_bf16x8(opnd[j]), as_bf16x8(pprev[c]), o[t]);
      } else {
        constexpr int js = kPV ? j - nPV : j;
        constexpr int cc = js / 2, st = js % 2;
        sn[st] = mfma32(as_bf16x8(opnd[j]), qf[cc], cc == 0 ? zero16 : sn[st]);
      }
    };

    // softmax state
    float mc[4], mt = 0.0f, m_new = 0.0f, alpha = 1.0f, negm = 0.0f;
    float x[32], pr[32];
    uint32_t w[16];
    // row sums of the tile: two chains, the first continuing the rescaled running sum
    float lt[2], le[2];
    auto E = [&](int f) -> float { return s[f >> 4][f & 15]; };
    // vector op k of the softmax
    auto op = [&](auto k_tag) {
      constexpr int k = decltype(k_tag)::value;
      if constexpr (k < nMask) {  // causal mask: keys past the row's position -> -inf
        constexpr int st = k >> 4, e = k & 15;
        constexpr int off = 32 * st + 16 * (e >> 3) + (e & 7);
        if (kbase + off > lim) s[st][e] = -INFINITY;
      } else if constexpr (k - nMask < 16) {  // four partial max chains of 8 scores
        constexpr int kk = k - nMask, c = kk % 4, u = kk / 4, f = 8 * c;
        if constexpr (u == 0) mc[c] = max3(E(f), E(f + 1), E(f + 2));
        if constexpr (u == 1) mc[c] = max3(mc[c], E(f + 3), E(f + 4));
        if constexpr (u == 2) mc[c] = max3(mc[c], E(f + 5), E(f + 6));
        if constexpr (u == 3) mc[c] = max3(mc[c], E(f + 7), E(f + 7));
      } else if constexpr (k - nMask == 16) {
        mt = max3(mc[0], mc[1], mc[2]);
      } else if constexpr (k - nMask == 17) {
        mt = max3(mt, mc[3], mc[3]);
      } else if constexpr (k - nMask == 18) {
        float x0, x1;
        lane_pair(mt, x0, x1);
        mt = max3(x0, x1, x1);
      } else if constexpr (k - nMask == 19) {
        mt *= csc;
      } else if constexpr (k - nMask == 20) {
        m_new = mt > m_ref + kRescaleSlack ? mt : m_ref;
      } else if constexpr (k - nMask == 21) {
        alpha = fast_exp2(m_ref - m_new);
      } else if constexpr (k - nMask == 22) {
        negm = -m_new;
        m_ref = m_new;
      } else if constexpr (k - nMask < kHead + 8 * kPerGroup) {
        constexpr int kk = k - nMask - kHead, g = kk / kPerGroup, r = kk % kPerGroup;
        if constexpr (r < 4) {
          x[4 * g + r] = fmaf(E(4 * g + r), csc, negm);
        } else if constexpr (r < 8) {
          pr[4 * g + r - 4] = fast_exp2(x[4 * g + r - 4]);
        } else {
          // then per word i = 2g, 2g+1: the bf16 pack, with kLse at once the exact fp32 sum
          // of its two probabilities (so they die here), and the rounded-weight row sums
          constexpr int rr = r - 8;
          constexpr int kind = kLse ? (rr < 4 ? rr % 2 : 2) : (rr < 2 ? 0 : 2);  // pack, exact, sum
          constexpr int i = 2 * g + (kLse ? (rr < 4 ? rr / 2 : rr - 4) : rr % 2);
          if constexpr (kind == 0) {
            w[i] = pack_bf16x2(pr[2 * i], pr[2 * i + 1]);
            pcur[i / 4][i % 4] = w[i];
            // keeps the word (and the FMAs and exponentials behind it) in this slot: the
            // compiler would otherwise sink them to where the next step first reads them
            asm volatile("" ::"v"(w[i]));
          } else if constexpr (kind == 1) {
            if constexpr (i == 0) le[0] = fmaf(l_exact, alpha, pr[0] + pr[1]);
            else if constexpr (i == 1) le[1] = pr[2] + pr[3];
            else le[i % 2] += pr[2 * i] + pr[2 * i + 1];
          } else {
            if constexpr (i == 0) lt[0] = add_bf16x2(w[0], l_part * alpha);
            else if constexpr (i == 1) lt[1] = add_bf16x2(w[1], 0.0f);
            else lt[i % 2] = add_bf16x2(w[i], lt[i % 2]);
          }
        }
      } else {
        l_part = lt[0] + lt[1];
        asm volatile("" ::"v"(l_part));
        if constexpr (kLse) {
          l_exact = le[0] + le[1];
          // like the words above: without it the exact sums (and every probability they
          // read) would be sunk into the next step, where l_exact is next used
          asm volatile("" ::"v"(l_exact));
        }
      }
    };

    static_for<kAhead>([&](auto j) { issue(j); });  // (with kPV: the operands in pre)
    static_for<nm>([&](auto m) {
      constexpr int mm = decltype(m)::value;
      issue(std::integral_constant<int, mm + kAhead>());
      mfma(m);
      constexpr int lo = mm * nOps / nm, hi = (mm + 1) * nOps / nm;
      static_for_range<lo, hi>([&](auto k) { op(k); });
      __builtin_amdgcn_sched_barrier(0);
    });
    return alpha;
  };

  // A wave whose 32 rows all lie past the block's tokens (the last, partial block of a
  // task) has nothing to compute: it only streams its rows of every K and V tile and
  // meets the workgroup at every barrier, in the same order as the computing waves (one
  // barrier after iteration -1, one after iteration 0 and one after each iteration
  // 1 .. ntiles - 1, each followed by the same group of loads into the same slots).
  // Its SIMD partner then runs alone.
  const bool wave_idle = wave * 32 >= it.ntok * G;
  if (wave_idle) {
    wait_vmem<S::kGroup + S::kDma>();
    tile_barrier();
    stream(k_lds0, v_lds2, 4, 2, fuse);
    wait_vmem<S::kGroup + S::kDma>();
    tile_barrier();
    stream(k_lds1, v_lds3, 5, 3, fuse);
    for (int i = 1; i < ntiles; ++i) {
      wait_vmem<S::kGroup + S::kDma>();
      tile_barrier();
      const int ks = (i + 1) & 3, vs = (i + 3) & 3;
      stream(ks == 0 ? k_lds0 : ks == 1 ? k_lds1 : ks == 2 ? k_lds2 : k_lds3,
             vs == 0 ? v_lds0 : vs == 1 ? v_lds1 : vs == 2 ? v_lds2 : v_lds3, i + 5, i + 3, fuse);
    }
    wait_vmem<0>();  // no transfer into LDS may outlive the workgroup
  } else {

  // ---- iteration -1: S(0), then K(4) / V(2) into the slots it leaves free ------------
  qk(k_lds0, sa);
  wait_vmem<S::kGroup + S::kDma>();  // V(0) and K(1) landed
  tile_barrier();
  stream(k_lds0, v_lds2, 4, 2, fuse);

  // ---- iteration 0: softmax(0) with S(1) ---------------------------------------------
  u32x4 pre_a[kAhead], pre_b[kAhead];  // first operands of odd / even iterations
  {
    float alpha;
    if (tbase >= n_full)
      alpha = block(std::false_type(), std::true_type(), tbase, sa, pa, pb, v_lds0, k_lds1, sb,
                    pre_b, v_lds0, pre_a);
    else
      alpha = block(std::false_type(), std::false_type(), tbase, sa, pa, pb, v_lds0, k_lds1, sb,
                    pre_b, v_lds0, pre_a);
    rescale(alpha);
  }
  wait_vmem<S::kGroup + S::kDma>();  // V(1) and K(2) landed
  tile_barrier();
  stream(k_lds1, v_lds3, 5, 3, fuse);

  // ---- iteration i >= 1: softmax(i) with P.V(i-1) and S(i+1) ----------------------------
  // Slots are fixed by i mod 4: S(i+1) reads K slot (i+1) mod 4, P.V(i-1) reads V slot
  // (i+3) mod 4 (its first operands were read by iteration i-1), the reads ahead for
  // iteration i+1 take V slot i mod 4, and after the barrier the slots just read receive
  // K(i+5) and V(i+3).  The S, P and read-ahead buffers alternate with the parity of i.
  auto step = [&](auto diag_tag, auto fuse_tag, int i, uint8_t* kb, uint8_t* vb,
                  const uint8_t* vb_next, f32x16(&s)[2], f32x16(&sn)[2],
                  const u32x4(&pprev)[4], u32x4(&pcur)[4], const u32x4(&pre)[kAhead],
                  u32x4(&pre_next)[kAhead]) __attribute__((always_inline)) {
    const float alpha = block(std::true_type(), diag_tag, tbase + i, s, pcur, pprev, vb, kb, sn,
                              pre, vb_next, pre_next);
    // the page ids of the next loads, fetched now so that the barrier hides their latency
    const PageRef kpg = page_ref(i + 5), vpg = page_ref(i + 3);
    rescale(alpha);
    wait_vmem<S::kGroup + S::kDma>();  // V(i+1) and K(i+2) landed
    tile_barrier();
    stream_pages(kb, vb, i + 5, i + 3, kpg, vpg, fuse_tag);
  };
  auto four = [&](auto diag_tag, auto fuse_tag, int i) __attribute__((always_inline)) {
    step(diag_tag, fuse_tag, i, k_lds2, v_lds0, v_lds1, sb, sa, pa, pb, pre_a, pre_b);
    step(diag_tag, fuse_tag, i + 1, k_lds3, v_lds1, v_lds2, sa, sb, pb, pa, pre_b, pre_a);
    step(diag_tag, fuse_tag, i + 2, k_lds0, v_lds2, v_lds3, sb, sa, pa, pb, pre_a, pre_b);
    step(diag_tag, fuse_tag, i + 3, k_lds1, v_lds3, v_lds0, sa, sb, pb, pa, pre_b, pre_a);
  };

  // Iterations 1 .. n_main - 1 see only tiles below the diagonal: four per loop trip,
  // unmasked, with every slot a compile-time array and no branch inside.  The rest (up to
  // three iterations left over by the four-way loop, and the tiles that cross the
  // diagonal, a few per item) run through the masked copy of the step, in the same slot
  // rotation.  (Choosing between a masked and an unmasked copy inside one step splits the
  // step at a branch, which costs the register allocator dearly.)
  //
  // With the fused append, the steps that stream only tiles below the prefix (K(i+5) under
  // P) run a copy of the step without the fused loads, so the long walk over the cached
  // history is the plain kernel's loop.
  const std::false_type plain, unmasked;
  const std::true_type masked;
  const int n_main = max(1, min(ntiles, n_full - tbase));
  int i = 1;
  if constexpr (kAppend) {
    const int first_new = P / 64 - tbase;  // first local tile holding a key >= P
    // a trip i .. i+3 is plain when its last stream, K(i+8), is still below first_new
    const int n_plain = min(n_main, first_new - 5);
    for (; i + 4 <= n_plain; i += 4) four(unmasked, plain, i);
  }
  for (; i + 4 <= n_main; i += 4) four(unmasked, fuse, i);
  for (; i + 4 <= ntiles; i += 4) four(masked, fuse, i);
  if (i < ntiles) {
    step(masked, fuse, i, k_lds2, v_lds0, v_lds1, sb, sa, pa, pb, pre_a, pre_b);
    if (i + 1 < ntiles) {
      step(masked, fuse, i + 1, k_lds3, v_lds1, v_lds2, sa, sb, pb, pa, pre_b, pre_a);
      if (i + 2 < ntiles)
        step(masked, fuse, i + 2, k_lds0, v_lds2, v_lds3, sb, sa, pa, pb, pre_a, pre_b);
    }
  }
  // P.V of the last tile n-1: V slot (n-1) mod 4, probabilities pa for even n-1
  const int last = tbase + ntiles - 1;
  switch ((ntiles - 1) & 3) {
    case 0: pv_tail(v_lds0, pa, last); break;
    case 1: pv_tail(v_lds1, pb, last); break;
    case 2: pv_tail(v_lds2, pa, last); break;
    default: pv_tail(v_lds3, pb, last); break;
  }
  wait_vmem<0>();  // no transfer into LDS may outlive the workgroup
  }  // computing waves

  // Fused append: this item's tokens' K/V rows into their pool slots (one chunk per item
  // writes).  No workgroup of this call reads those slots -- keys at or past P come from
  // the new rows -- so the stores need no ordering with anything else in the call.
  if (kAppend && (!kSplit || split <= 0)) {
    uint16_t* kp = const_cast<uint16_t*>(a.k_pool);
    uint16_t* vp = const_cast<uint16_t*>(a.v_pool);
    for (int idx = tid; idx < it.ntok * S::kNG; idx += kThreads) {
      const int row = idx / S::kNG, g = idx - row * S::kNG;
      const int pos = P + it.tok0 + row;
      const int32_t page = bt[pos / kPage];
      if (page < 0 || page >= a.num_pages) {
        bad_page = true;
        continue;
      }
      const int64_t src = (new_row0 + (int64_t)(it.tok0 + row) * a.num_kv_heads) * D + 8 * g;
      const int64_t dst =
          (((int64_t)page * a.num_kv_heads + it.kv_head) * kPage + pos % kPage) * D + 8 * g;
      store_u32x4(kp + dst, load_u32x4(a.k_new + src));
      store_u32x4(vp + dst, load_u32x4(a.v_new + src));
    }
  }

  if constexpr (kAppend) {  // the pool writes test page ids per lane
    if ((__builtin_amdgcn_ballot_w64(bad_page) != 0 || bad_tile) && lane == 0)
      atomicOr(a.error_flags, 1);
  } else {
    if (bad_tile && lane == 0) atomicOr(a.error_flags, 1);
  }
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

}  // namespace kern
}  // namespace tide
