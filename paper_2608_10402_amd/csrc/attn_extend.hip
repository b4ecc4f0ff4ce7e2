// Extend attention over the paged KV pool (and full prefill, which is the same kernel
// with prefix 0): the compute of a resumed task that kept its cache (TideRL,
// Continuous Task Batching, Sections 4 and 4.2) and of the recompute that an evicted
// cache forces (challenge C1, Section 2.2).
//
// Method: FlashAttention-2-style streaming softmax (Dao 2023; online softmax of Milakov
// & Gimelshein 2018) over K/V gathered page by page (PagedAttention, Kwon et al. 2023),
// laid out for CDNA4:
//   * A workgroup owns one (task, kv head, block of tokens) item.  Its NW*32 query rows
//     are the (token, head) pairs of the block for every query head of the kv head, so
//     each K/V tile staged in LDS serves all G grouped heads at once.
//   * Each wave computes S^T = K.Q^T for its 32 rows with v_mfma_f32_32x32x16_bf16:
//     keys are the MFMA rows, queries the columns, so every lane owns one query row and
//     its softmax statistics need only one cross-lane exchange (lanes l and l^32).
//   * Key rows are loaded in the perm32 order, which leaves each lane holding runs of 8
//     consecutive keys: the probabilities convert straight into the B operand of the
//     O^T += V^T.P^T MFMA without any shuffle.  V pages are stored transposed in the
//     pool (head-dim major, 16 token slots contiguous), so V^T operands are plain
//     16-byte LDS reads.
//   * Scores are kept in base-2 units (sm_scale * log2 e folded in) and exponentiated
//     with v_exp_f32.  The running max is only raised when a tile exceeds it by more
//     than kRescaleSlack, so the O rescale is skipped on almost every tile.
//   * Causal masking is applied only on the tiles that cross the diagonal, and V slots
//     at or beyond the task's length are zeroed while staging so that NaN/Inf garbage in
//     unused pool slots can never reach the output.
#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace {

template <int D, int NW>
struct Shape {
  static constexpr int kThreads = NW * 64;
  static constexpr int kKeys = kExtendKeyTile;          // 64 keys = 4 pages per tile
  static constexpr int kPages = kKeys / kPage;
  static constexpr int kKPitch = D + 8;                 // padded K row (bf16 elements)
  static constexpr int kKTile = kKeys * kKPitch;
  static constexpr int kVTile = kPages * D * kPage;     // 4 transposed pages
  static constexpr int kKChunks = kKeys * D / 8;        // 16-byte chunks per tile
  static constexpr int kVChunks = kVTile / 8;
  static constexpr int kKPer = kKChunks / kThreads;
  static constexpr int kVPer = kVChunks / kThreads;
  static_assert(kKChunks % kThreads == 0 && kVChunks % kThreads == 0, "tile split");
};

template <int D, int NW>
struct Staged {
  u32x4 k[Shape<D, NW>::kKPer];
  u32x4 v[Shape<D, NW>::kVPer];
};

// Keep only the first n (0..8) bf16 elements of a 16-byte chunk.
__device__ __forceinline__ u32x4 keep_first(u32x4 x, int n) {
  u32x4 r;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t lo = (2 * w < n) ? 0x0000FFFFu : 0u;
    const uint32_t hi = (2 * w + 1 < n) ? 0xFFFF0000u : 0u;
    r[w] = x[w] & (lo | hi);
  }
  return r;
}

template <int D, int NW>
__device__ __forceinline__ void load_tile(Staged<D, NW>& st, const ExtendArgs& a,
                                          const int32_t* bt_row, int npages, int seq_len,
                                          int kv_head, int tile, int tid) {
  using S = Shape<D, NW>;
  int64_t base[S::kPages];  // element offset of (page, kv_head) block, or -1
#pragma unroll
  for (int pi = 0; pi < S::kPages; ++pi) {
    const int lp = tile * S::kPages + pi;
    int64_t b = -1;
    if (lp < npages) {
      const int32_t p = bt_row[lp];
      if (p >= 0 && p < a.num_pages) {
        b = ((int64_t)p * a.num_kv_heads + kv_head) * (int64_t)(kPage * D);
      } else if (tid == 0) {
        atomicOr(a.error_flags, 1);
      }
    }
    base[pi] = b;
  }
#pragma unroll
  for (int i = 0; i < S::kKPer; ++i) {
    const int c = tid + i * S::kThreads;
    const int key = c / (D / 8), part = c % (D / 8);
    const int64_t b = base[key / kPage];
    st.k[i] = b >= 0 ? load_u32x4(a.k_pool + b + (key % kPage) * D + part * 8) : zero_u32x4();
  }
  const bool tail = (tile + 1) * S::kKeys > seq_len;
#pragma unroll
  for (int i = 0; i < S::kVPer; ++i) {
    const int c = tid + i * S::kThreads;
    const int pi = c / (D * 2);
    const int off = (c % (D * 2)) * 8;  // within the page's [D][16] block
    const int64_t b = base[pi];
    u32x4 x = b >= 0 ? load_u32x4(a.v_pool + b + off) : zero_u32x4();
    if (tail) {
      const int key0 = tile * S::kKeys + pi * kPage + (off & (kPage - 1));
      x = keep_first(x, seq_len - key0);
    }
    st.v[i] = x;
  }
}

template <int D, int NW>
__device__ __forceinline__ void store_tile(const Staged<D, NW>& st, uint16_t* k_lds,
                                           uint16_t* v_lds, int tid) {
  using S = Shape<D, NW>;
#pragma unroll
  for (int i = 0; i < S::kKPer; ++i) {
    const int c = tid + i * S::kThreads;
    const int key = c / (D / 8), part = c % (D / 8);
    store_u32x4(k_lds + key * S::kKPitch + part * 8, st.k[i]);
  }
#pragma unroll
  for (int i = 0; i < S::kVPer; ++i) {
    const int c = tid + i * S::kThreads;
    store_u32x4(v_lds + c * 8, st.v[i]);
  }
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void extend_attn_kernel(ExtendArgs a) {
  using S = Shape<D, NW>;
  constexpr int kDC = D / 16;  // 16-wide head-dim chunks of the QK^T contraction
  constexpr int kDT = D / 32;  // 32-row head-dim tiles of O^T
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][S::kKTile];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][S::kVTile];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int q = lane & 31, h = lane >> 5;

  const ExtendItem it = a.items[blockIdx.x];
  const TaskDesc td = a.tasks[it.task];
  const int P = td.prefix;
  const int seq_len = td.prefix + td.extend;
  const int npages = (seq_len + kPage - 1) / kPage;
  const int32_t* bt_row = a.block_table + (int64_t)it.task * a.bt_stride;
  const int G = a.group;

  // this lane's query row: (token tk of the block, head j of the group)
  const int r = wave * 32 + q;
  const int tk = r / G, j = r - (r / G) * G;
  const bool row_valid = tk < it.ntok;
  const int lim = row_valid ? P + it.tok0 + tk : -1;  // last visible key position
  const int64_t qrow = (int64_t)(td.row_start + it.tok0 + tk) * a.num_q_heads +
                       it.kv_head * G + j;

  bf16x8 qf[kDC];
#pragma unroll
  for (int c = 0; c < kDC; ++c)
    qf[c] = as_bf16x8(row_valid ? load_u32x4(a.q + qrow * D + 16 * c + 8 * h) : zero_u32x4());

  const int kend = P + it.tok0 + it.ntok;            // keys needed by the last row
  const int ntiles = (kend + S::kKeys - 1) / S::kKeys;
  const int n_full = (P + it.tok0 + 1) / S::kKeys;   // tiles every row sees completely

  f32x16 o[kDT];
#pragma unroll
  for (int t = 0; t < kDT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_ref = kNoMax, l_part = 0.0f;

  Staged<D, NW> stg;
  load_tile<D, NW>(stg, a, bt_row, npages, seq_len, it.kv_head, 0, tid);
  store_tile<D, NW>(stg, k_lds[0], v_lds[0], tid);
  __syncthreads();

  const int krow = perm32(q);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    const bool more = tile + 1 < ntiles;
    if (more) load_tile<D, NW>(stg, a, bt_row, npages, seq_len, it.kv_head, tile + 1, tid);

    const uint16_t* kl = k_lds[buf];
    const uint16_t* vl = v_lds[buf];

    // S^T for the two 32-key halves of the tile
    f32x16 s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[st][e] = 0.0f;
#pragma unroll
      for (int c = 0; c < kDC; ++c) {
        const bf16x8 kf =
            as_bf16x8(load_u32x4(kl + (st * 32 + krow) * S::kKPitch + 16 * c + 8 * h));
        s[st] = mfma32(kf, qf[c], s[st]);
      }
    }

    // scale, mask, tile max
    const bool masked = tile >= n_full;
    const int k0 = tile * S::kKeys;
    float mt = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float x = s[st][e] * a.scale_log2;
        if (masked) {
          const int key = k0 + 32 * st + 16 * (e >> 3) + 8 * h + (e & 7);
          x = key <= lim ? x : -INFINITY;
        }
        s[st][e] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, xor_shfl(mt, 32));
    if (__any(mt > m_ref + kRescaleSlack)) {
      const float m_new = fmaxf(m_ref, mt);
      const float alpha = fast_exp2(m_ref - m_new);
      l_part *= alpha;
#pragma unroll
      for (int t = 0; t < kDT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
      m_ref = m_new;
    }

    // probabilities -> bf16 B operands, 8 consecutive keys per lane
    bf16x8 pb[2][2];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(s[st][8 * m + 2 * e] - m_ref);
          const float p1 = fast_exp2(s[st][8 * m + 2 * e + 1] - m_ref);
          l_part += p0 + p1;
          w[e] = pack_bf16x2(p0, p1);
        }
        pb[st][m] = as_bf16x8(w);
      }

    // O^T += V^T . P^T, 16 keys (one page) per MFMA
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const uint16_t* vp = vl + (2 * st + m) * D * kPage + 8 * h;
#pragma unroll
        for (int t = 0; t < kDT; ++t) {
          const bf16x8 vf = as_bf16x8(load_u32x4(vp + (32 * t + krow) * kPage));
          o[t] = mfma32(vf, pb[st][m], o[t]);
        }
      }

    if (more) store_tile<D, NW>(stg, k_lds[buf ^ 1], v_lds[buf ^ 1], tid);
    __syncthreads();
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
    if (a.lse && h == 0) a.lse[qrow] = (m_ref + __log2f(l_tot)) * kLn2;
  }
}

template <int D, int NW>
hipError_t launch(const ExtendArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((extend_attn_kernel<D, NW>), dim3(a.num_items), dim3(NW * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_extend(const ExtendArgs& a, int head_dim, int waves, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  if (head_dim == 128 && waves == 4) return launch<128, 4>(a, stream);
  if (head_dim == 64 && waves == 4) return launch<64, 4>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
