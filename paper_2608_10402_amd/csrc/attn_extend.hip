// Extend attention over the paged KV pool (and full prefill, which is the same kernel
// with prefix 0): the compute of a resumed task that kept its cache (TideRL,
// Continuous Task Batching, Sections 4 and 4.2) and of the recompute that an evicted
// cache forces (challenge C1, Section 2.2).
//
// Method: FlashAttention-2-style streaming softmax (Dao 2023; online softmax of Milakov
// & Gimelshein 2018) over K/V gathered page by page (PagedAttention, Kwon et al. 2023),
// laid out for CDNA4:
//   * A workgroup (4 waves) owns one (task, kv head, block of tokens) item.  Its 128
//     query rows are the (token, head) pairs of the block for every query head of the kv
//     head, so each K/V tile in LDS serves all G grouped heads at once.
//   * K/V tiles of 64 keys (4 pages) go from HBM straight into LDS with
//     global_load_lds_dwordx4 (no staging registers); wave w fetches page w of the tile.
//     Two LDS buffers: the next tile streams in while the current one is used.
//   * Each wave computes S^T = K.Q^T for its 32 rows with v_mfma_f32_32x32x16_bf16:
//     keys are the MFMA rows, queries the columns, so every lane owns one query row and
//     its softmax statistics need one cross-lane exchange (lanes l and l^32).
//   * Key rows are read in the perm32 order, which leaves each lane holding runs of 8
//     consecutive keys: the probabilities convert straight into the B operand of the
//     O^T += V^T.P^T MFMA with no shuffle.  V pages are stored transposed in the pool
//     (head-dim major, 16 token slots contiguous), so V^T operands are plain 16-byte LDS
//     reads.  K rows are XOR-swizzled by 16-byte granule in LDS so that the 64 lanes of an
//     operand read hit distinct banks; V^T rows swap their 16-byte halves every 8 rows.
//   * Scores stay raw until one FMA applies sm_scale*log2(e) and subtracts the running
//     max before v_exp_f32.  The running max is only raised when a tile exceeds it by
//     more than kRescaleSlack, so the O rescale is skipped on almost every tile.
//   * Causal masking is applied only on tiles that cross the diagonal.  V slots at or
//     beyond the task's length (the last tile) are zeroed in LDS before use, so NaN/Inf
//     garbage in unused pool slots can never reach the output.
//   * At most 256 registers per lane, so two workgroups share a CU and one's softmax
//     overlaps the other's matrix work.
#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWaves = 4;
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
  static_assert(kDma >= 1 && kRowsPerDma * kRowBytes == 1024, "page split");
};

// Swizzled position of granule g in K row r.
template <int D>
__device__ __forceinline__ int kswz(int r, int g) {
  return g ^ ((r / ES<D>::kRB) % ES<D>::kNG);
}

// Position (0/1) of 16-byte half `hh` of V^T row d in LDS: rows d and d+8 share banks,
// so the halves of rows with bit 3 set are swapped.
__device__ __forceinline__ int vswz(int d, int hh) { return hh ^ ((d >> 3) & 1); }

__device__ __forceinline__ void wait_all_vmem() {
  // s_waitcnt vmcnt(0) (gfx9 encoding: expcnt and lgkmcnt left at their maxima)
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

template <int D>
struct Ctx {
  const uint8_t* k_pool;
  const uint8_t* v_pool;
  int32_t* error_flags;
  int64_t num_pages;
  int num_kv_heads;
  const int32_t* bt_row;
  int npages;
  int seq_len;
  int kv_head;
  int wave;
  int lane;
  uint32_t k_dma_off[ES<D>::kDma];  // this lane's source offset inside a K page, per transfer
  uint32_t v_dma_off[ES<D>::kDma];  // same for the V^T page

  // Block-table word of this wave's page (page `wave`) of tile `tile`, loaded as a vector
  // value: it is issued one tile ahead and only read after the next vmcnt(0), so the
  // memory round trip overlaps a whole tile of compute instead of stalling the issue.
  __device__ __forceinline__ int32_t fetch_page(int tile) const {
    const int lp = tile * 4 + wave;
    return lp < npages ? bt_row[lp] : 0;
  }

  // Issue this wave's share of a tile, whose page id `word` came from fetch_page().
  __device__ __forceinline__ void issue_tile(int32_t word, uint8_t* kb, uint8_t* vb) const {
    using S = ES<D>;
    // One word for the whole wave: kept scalar, as is all the address math below.
    const int32_t p = __builtin_amdgcn_readfirstlane(word);
    const bool bad = p < 0 || p >= num_pages;
    const int64_t page = bad ? 0 : p;
    if (bad && lane == 0) atomicOr(error_flags, 1);
    // Pages past the sequence (and invalid ids) are read from page 0, which always
    // exists; their keys are masked and their V slots zeroed before use.
    const int64_t blk = (page * num_kv_heads + kv_head) * (int64_t)S::kPageBytes;
    const uint8_t* kg = k_pool + blk;
    const uint8_t* vg = v_pool + blk;
    uint8_t* kd = kb + wave * S::kPageBytes;
    uint8_t* vd = vb + wave * S::kPageBytes;
#pragma unroll
    for (int i = 0; i < S::kDma; ++i) {
      __builtin_amdgcn_global_load_lds(kg + k_dma_off[i], kd + i * 1024, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vg + v_dma_off[i], vd + i * 1024, 16, 0, 0);
    }
  }
};

// Zero the V^T slots of keys >= seq_len in a tile (only the last tile of an item).
template <int D>
__device__ __forceinline__ void zero_tail(uint8_t* vb, int k0, int seq_len, int tid) {
  using S = ES<D>;
  for (int row = tid; row < 4 * D; row += kThreads) {
    const int pi = row / D, d = row % D;
    const int nvalid = seq_len - (k0 + pi * kPage);
    if (nvalid >= kPage) continue;
    uint8_t* r = vb + pi * S::kPageBytes + d * (kPage * 2);
    for (int s = nvalid < 0 ? 0 : nvalid; s < kPage; ++s)
      *reinterpret_cast<uint16_t*>(r + vswz(d, s >> 3) * 16 + (s & 7) * 2) = 0;
  }
}

// kLse: also keep the exact fp32 sum of the probabilities, so the returned log-sum-exp is
// the true one; the output itself is normalised by the sum of the bf16-rounded weights
// that the P.V product used.
template <int D, bool kLse>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void extend_attn_kernel(ExtendArgs a) {
  using S = ES<D>;
  constexpr int kDC = D / 16;  // 16-wide head-dim chunks of QK^T
  constexpr int kDT = D / 32;  // 32-row head-dim tiles of O^T
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds1[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds0[S::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds1[S::kTileBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane & 31, h = lane >> 5;

  const ExtendItem it = a.items[blockIdx.x];
  if (it.ntok == 0) return;  // padding slot of the XCD-interleaved work list
  const TaskDesc td = a.tasks[it.task];
  const int P = td.prefix;
  const int seq_len = td.prefix + td.extend;
  const int G = a.group;

  Ctx<D> c;
  c.k_pool = reinterpret_cast<const uint8_t*>(a.k_pool);
  c.v_pool = reinterpret_cast<const uint8_t*>(a.v_pool);
  c.error_flags = a.error_flags;
  c.num_pages = a.num_pages;
  c.num_kv_heads = a.num_kv_heads;
  c.bt_row = a.block_table + (int64_t)it.task * a.bt_stride;
  c.npages = (seq_len + kPage - 1) / kPage;
  c.seq_len = seq_len;
  c.kv_head = it.kv_head;
  c.wave = wave;
  c.lane = lane;
#pragma unroll
  for (int i = 0; i < S::kDma; ++i) {
    const int r = i * S::kRowsPerDma + lane / S::kNG;  // row inside the page (== tile row mod 16)
    const int g = kswz<D>(r, lane % S::kNG);
    c.k_dma_off[i] = (uint32_t)(r * S::kRowBytes + g * 16);
    const int d = i * 32 + lane / 2;  // V^T row (head-dim entry) this lane's granule lands in
    c.v_dma_off[i] = (uint32_t)(d * (kPage * 2) + vswz(d, lane & 1) * 16);
  }

  // start streaming tile 0 before anything else
  c.issue_tile(c.fetch_page(0), k_lds0, v_lds0);
  int32_t next_page = c.fetch_page(1);  // page id of the tile the next step streams in

  // this lane's query row: (token tk of the block, head j of the group)
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

  // per-lane LDS byte offsets of the MFMA operands
  const int krow = perm32(q);
  int k_rd[kDC];
#pragma unroll
  for (int cc = 0; cc < kDC; ++cc) k_rd[cc] = krow * S::kRowBytes + kswz<D>(krow, 2 * cc + h) * 16;
  const int v_rd = krow * (kPage * 2) + vswz(krow, h) * 16;

  const int kend = P + it.tok0 + it.ntok;           // keys needed by the last row
  const int ntiles = (kend + 63) / 64;
  const int n_full = (P + it.tok0 + 1) / 64;        // tiles every row sees completely
  const float csc = a.scale_log2;

  f32x16 o[kDT];
#pragma unroll
  for (int t = 0; t < kDT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;

  auto compute = [&](const uint8_t* kb, const uint8_t* vb, int tile) {
    f32x16 s[2];
    {
      u32x4 kf[2][kDC];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int cc = 0; cc < kDC; ++cc)
          kf[st][cc] = load_u32x4(kb + st * 32 * S::kRowBytes + k_rd[cc]);
#pragma unroll
      for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int e = 0; e < 16; ++e) s[st][e] = 0.0f;
#pragma unroll
        for (int cc = 0; cc < kDC; ++cc) s[st] = mfma32(as_bf16x8(kf[st][cc]), qf[cc], s[st]);
      }
      // Keep kDC operand reads in flight ahead of the MFMAs: all reads of the first
      // half, then MFMA/read pairs, then the last MFMAs.
      __builtin_amdgcn_sched_group_barrier(0x100, kDC, 0);
#pragma unroll
      for (int i = 0; i < kDC; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, kDC, 0);
    }
    if (tile >= n_full) {  // diagonal / tail tile: hide keys past this row's position
      const int kbase = tile * 64 + 8 * h;
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
    mt = fmaxf(mt, xor_shfl(mt, 32)) * csc;
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
    float lt = 0.0f, le = 0.0f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(fmaf(s[st][8 * m + 2 * e], csc, negm));
          const float p1 = fast_exp2(fmaf(s[st][8 * m + 2 * e + 1], csc, negm));
          w[e] = pack_bf16x2(p0, p1);
          lt = add_bf16x2(w[e], lt);
          if (kLse) le += p0 + p1;
        }
        const bf16x8 pb = as_bf16x8(w);
        const uint8_t* vp = vb + (2 * st + m) * S::kPageBytes + v_rd;
#pragma unroll
        for (int t = 0; t < kDT; ++t)
          o[t] = mfma32(as_bf16x8(load_u32x4(vp + t * 1024)), pb, o[t]);
      }
    l_part += lt;  // short dot2 chains per tile, IEEE adds across tiles
    if (kLse) l_exact += le;
  };

  auto step = [&](int tile, uint8_t* kb, uint8_t* vb, uint8_t* kn, uint8_t* vn) {
    wait_all_vmem();
    __syncthreads();  // tile landed for every wave; the other buffer is free again
    if ((tile + 1) * 64 > seq_len) {
      zero_tail<D>(vb, tile * 64, seq_len, tid);
      __syncthreads();
    }
    if (tile + 1 < ntiles) {
      c.issue_tile(next_page, kn, vn);
      next_page = c.fetch_page(tile + 2);
    }
    compute(kb, vb, tile);
  };

  for (int tile = 0; tile < ntiles; tile += 2) {
    step(tile, k_lds0, v_lds0, k_lds1, v_lds1);
    if (tile + 1 < ntiles) step(tile + 1, k_lds1, v_lds1, k_lds0, v_lds0);
  }

  const float l_tot = l_part + xor_shfl(l_part, 32);
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
      const float l_ex = l_exact + xor_shfl(l_exact, 32);
      if (h == 0) a.lse[qrow] = (m_ref + __log2f(l_ex)) * kLn2;
    }
  }
}

template <int D>
hipError_t launch(const ExtendArgs& a, hipStream_t stream) {
  if (a.lse)
    hipLaunchKernelGGL((extend_attn_kernel<D, true>), dim3(a.num_items), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((extend_attn_kernel<D, false>), dim3(a.num_items), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

// Both variants of each head size are instantiated explicitly: the host pass otherwise
// emits the launch stub of only one of two specialisations that differ in the bool.
template __global__ void extend_attn_kernel<128, false>(ExtendArgs);
template __global__ void extend_attn_kernel<128, true>(ExtendArgs);
template __global__ void extend_attn_kernel<64, false>(ExtendArgs);
template __global__ void extend_attn_kernel<64, true>(ExtendArgs);

}  // namespace kern

hipError_t launch_extend(const ExtendArgs& a, int head_dim, int waves, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (waves != kern::kWaves) return hipErrorInvalidValue;
  if (head_dim == 128) return kern::launch<128>(a, stream);
  if (head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
