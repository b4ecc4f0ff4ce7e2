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
//   * Operands go straight from HBM into MFMA registers (no LDS): for S^T = K.Q^T a lane
//     loads 16 contiguous bytes of one key row; for O^T += V^T.P^T it loads 16 bytes of
//     a transposed V page (8 consecutive token slots of one head-dim entry).  Key rows
//     are assigned so that each lane's probabilities are those 8 slots, so P never moves
//     between lanes.
//   * The next 32-key step is loaded while the current one is computed.
//   * Partial (o, m, l) per split go to the workspace; a second small kernel merges them.
#include "kernels.h"
#include "tide_device.h"

namespace tide {
namespace kern {

constexpr int kWavesPerBlock = 4;

template <int D>
struct DecodeRegs {
  u32x4 k[2][D / 32];  // two 16-key S tiles x head-dim chunks of 32
  u32x4 v[D / 16];     // V^T operands, one per 16-row head-dim tile
};

template <int D>
__device__ __forceinline__ void load_step(DecodeRegs<D>& r, const DecodeArgs& a,
                                          const int32_t* bt_row, int npages, int kv_len,
                                          int kv_head, int k, int lane) {
  const int lp0 = k / kPage;
  int64_t base[2];
#pragma unroll
  for (int pi = 0; pi < 2; ++pi) {
    const int lp = lp0 + pi;
    int64_t b = -1;
    if (lp < npages) {
      const int32_t p = bt_row[lp];
      if (p >= 0 && p < a.num_pages) {
        b = ((int64_t)p * a.num_kv_heads + kv_head) * (int64_t)(kPage * D);
      } else if (lane == 0) {
        atomicOr(a.error_flags, 1);
      }
    }
    base[pi] = b;
  }
  const int row = lane & 15, grp = lane >> 4;
  // K rows: S tile t, MFMA row `row` holds key 8*(row/4) + 4*t + row%4 of the 32-key step
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int key = 8 * (row >> 2) + 4 * t + (row & 3);
    const int64_t b = base[key >> 4];
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
      r.k[t][c] = b >= 0 ? load_u32x4(a.k_pool + b + (key & 15) * D + 32 * c + 8 * grp)
                         : zero_u32x4();
  }
  // V^T: lane group grp holds keys 8*grp .. 8*grp+7 = page grp/2, slots 8*(grp&1) ..
  const int64_t vb = base[grp >> 1];
  const int slot0 = 8 * (grp & 1);
  const int nvalid = kv_len - (k + 8 * grp);
#pragma unroll
  for (int t = 0; t < D / 16; ++t) {
    u32x4 x = vb >= 0 ? load_u32x4(a.v_pool + vb + (16 * t + row) * kPage + slot0)
                      : zero_u32x4();
    if (nvalid < 8) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = (2 * w < nvalid) ? 0x0000FFFFu : 0u;
        const uint32_t hi = (2 * w + 1 < nvalid) ? 0xFFFF0000u : 0u;
        x[w] &= (lo | hi);
      }
    }
    r.v[t] = x;
  }
}

template <int D>
__global__ __launch_bounds__(kWavesPerBlock * 64) void decode_split_kernel(DecodeArgs a) {
  const int lane = threadIdx.x & 63;
  const int item_id = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (item_id >= a.num_items) return;  // whole wave exits; no block-level barrier below
  const DecodeItem it = a.items[item_id];
  const TaskDesc td = a.tasks[it.task];
  const int kv_len = td.prefix + td.extend;
  const int npages = (kv_len + kPage - 1) / kPage;
  const int32_t* bt_row = a.block_table + (int64_t)it.task * a.bt_stride;
  const int G = a.group;
  const int col = lane & 15, grp = lane >> 4;

  // Q^T operand: column col = query head kv_head*G + col (zero when col >= G)
  bf16x8 qf[D / 32];
  const int64_t qrow = (int64_t)td.row_start * a.num_q_heads + it.kv_head * G + col;
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
    qf[c] = as_bf16x8(col < G ? load_u32x4(a.q + qrow * D + 32 * c + 8 * grp) : zero_u32x4());

  const int kbeg = it.k_begin;
  const int kend = min(kv_len, kbeg + a.chunk);

  f32x4 o[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t) o[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_ref = kNoMax, l_part = 0.0f, l_exact = 0.0f;

  DecodeRegs<D> cur, nxt;
  load_step<D>(cur, a, bt_row, npages, kv_len, it.kv_head, kbeg, lane);
  for (int k = kbeg; k < kend; k += kDecodeStep) {
    const bool more = k + kDecodeStep < kend;
    if (more) load_step<D>(nxt, a, bt_row, npages, kv_len, it.kv_head, k + kDecodeStep, lane);

    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < D / 32; ++c) s[t] = mfma16(as_bf16x8(cur.k[t][c]), qf[c], s[t]);
    }
    // s[t][e] is key k + 8*grp + 4*t + e of query head `col`
    float mt = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float x = s[t][e] * a.scale_log2;
        x = (k + 8 * grp + 4 * t + e < kv_len) ? x : -INFINITY;
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
    for (int t = 0; t < D / 16; ++t) o[t] = mfma16(as_bf16x8(cur.v[t]), pb, o[t]);
    if (more) cur = nxt;
  }

  float l_tot = l_part + xor_shfl(l_part, 16);
  l_tot += xor_shfl(l_tot, 32);
  float l_ex = l_exact + xor_shfl(l_exact, 16);
  l_ex += xor_shfl(l_ex, 32);
  if (col < G) {
    const int64_t slot =
        ((int64_t)it.task * a.num_q_heads + it.kv_head * G + col) * a.max_splits + it.split;
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, xor_shfl(v, m));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += xor_shfl(v, m);
  return v;
}

// One wave per (task, query head): combine the task's split partials.  Lane s owns split
// s for the statistics (max, weights); the partial outputs are then accumulated with
// every lane covering D/64 head-dim entries and the weights broadcast across the wave.
template <int D>
__global__ __launch_bounds__(kWavesPerBlock * 64) void decode_merge_kernel(DecodeArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (row >= (int64_t)a.num_tasks * a.num_q_heads) return;
  const int task = (int)(row / a.num_q_heads);
  const int nsplit = a.tasks[task].aux;
  const float* ml = a.part_ml + row * a.max_splits * 4;
  const float* po = a.part_o + row * a.max_splits * D;
  constexpr int kPer = D / 64;

  float mx = kNoMax;
  for (int s = lane; s < nsplit; s += 64) mx = fmaxf(mx, ml[4 * s]);
  mx = wave_max(mx);

  float acc[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) acc[i] = 0.0f;
  float l_round = 0.0f, l_ex = 0.0f;
  for (int s0 = 0; s0 < nsplit; s0 += 64) {
    const int s = s0 + lane;
    float wgt = 0.0f;
    if (s < nsplit) {
      const f32x4 st = *reinterpret_cast<const f32x4*>(ml + 4 * s);
      wgt = fast_exp2(st[0] - mx);
      l_round += wgt * st[1];
      l_ex += wgt * st[2];
    }
    const int n = min(64, nsplit - s0);
#pragma unroll 4
    for (int i = 0; i < n; ++i) {
      const float wi = __shfl(wgt, i, 64);
      const float* src = po + (int64_t)(s0 + i) * D + kPer * lane;
#pragma unroll
      for (int k = 0; k < kPer; ++k) acc[k] += wi * src[k];
    }
  }
  l_round = wave_sum(l_round);
  const float inv = 1.0f / l_round;
  uint16_t* orow = a.out + row * D;
  if (kPer == 2) {
    *reinterpret_cast<uint32_t*>(orow + 2 * lane) = pack_bf16x2(acc[0] * inv, acc[kPer - 1] * inv);
  } else {
    const uint32_t w = pack_bf16x2(acc[0] * inv, 0.0f);
    orow[lane] = (uint16_t)(w & 0xFFFFu);
  }
  if (a.lse) {
    l_ex = wave_sum(l_ex);
    if (lane == 0) a.lse[row] = (mx + __log2f(l_ex)) * kLn2;
  }
}

template <int D>
hipError_t launch(const DecodeArgs& a, hipStream_t stream) {
  if (a.num_items > 0) {
    const int blocks = (a.num_items + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((decode_split_kernel<D>), dim3(blocks), dim3(kWavesPerBlock * 64), 0,
                       stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t rows = (int64_t)a.num_tasks * a.num_q_heads;
  if (rows > 0) {
    const int blocks = (int)((rows + kWavesPerBlock - 1) / kWavesPerBlock);
    hipLaunchKernelGGL((decode_merge_kernel<D>), dim3(blocks), dim3(kWavesPerBlock * 64), 0,
                       stream, a);
  }
  return hipGetLastError();
}

}  // namespace kern

hipError_t launch_decode(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 128) return kern::launch<128>(a, stream);
  if (head_dim == 64) return kern::launch<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tide
