// Device helpers for the gfx950 kernels: vector types, bf16 packing, MFMA wrappers and
// the lane-permutation that makes MFMA outputs feed the next MFMA directly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tide_common.h"

namespace tide {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLog2e = 1.44269504088896340736f;
// Running-max sentinel: finite so that exp2(m_old - m_new) never sees (-inf) - (-inf).
constexpr float kNoMax = -1.0e30f;
// A row's reference max is only raised when the tile max exceeds it by more than this
// (base-2 units).  Unnormalised weights then stay <= 2^8, far from fp32/bf16 limits,
// and the accumulator rescale is skipped on almost every tile.
constexpr float kRescaleSlack = 8.0f;

typedef const __attribute__((address_space(4))) int32_t const_i32;

// Block-table word `idx` of a row, read through the constant address space: the table is
// read-only during a kernel, so a wave-uniform index becomes a scalar load (counted by
// lgkmcnt, so waiting for it never waits for outstanding vector loads).
__device__ __forceinline__ int32_t load_page_id(const int32_t* row, int idx) {
  return ((const_i32*)row)[idx];
}

__device__ __forceinline__ u32x4 load_u32x4(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ void store_u32x4(void* p, u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 zero_u32x4() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return z;
}

// Two fp32 values -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// acc + lo + hi of a packed bf16 pair (v_dot2c_f32_bf16 against (1, 1)).  Summing the
// rounded probabilities keeps the softmax denominator consistent with the bf16 weights
// the P.V product actually uses, at half a VALU instruction per probability.
__device__ __forceinline__ float add_bf16x2(uint32_t packed, float acc) {
  const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1.0, 1.0)
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, packed), one, acc, false);
}

__device__ __forceinline__ float xor_shfl(float v, int mask) {
  return __shfl_xor(v, mask, 64);
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

// One wave combines n >= 1 split partials of one (row, query head), the split-K merge of
// flash decoding: partial s holds, at ml + s * ml_stride, its running max m_s (base-2
// units), the sum of its bf16-rounded weights and their exact fp32 sum, and at
// po + s * po_stride its unnormalised output.  With M = max m_s and w_s = 2^(m_s - M) the
// row is sum_s w_s o_s / sum_s w_s l_s, written as bf16 to orow; when lse_out is non-null
// it receives ln(sum_s w_s l_exact_s) + M ln 2.  Lane s owns split s for the statistics;
// the outputs are accumulated with every lane covering D/64 entries.
template <int D>
__device__ __forceinline__ void merge_partials(const float* ml, int64_t ml_stride, const float* po,
                                               int64_t po_stride, int n, uint16_t* orow,
                                               float* lse_out) {
  const int lane = threadIdx.x & 63;
  constexpr int kPer = D / 64;
  constexpr int kFew = 16;
  if (n <= kFew) {
    // Up to kFew splits: the statistics and every partial this lane needs are loaded
    // before any arithmetic, so the wave waits for one memory round trip, not two.  The
    // sums run in the same order as below, so both paths give identical results.
    f32x4 st = {kNoMax, 0.0f, 0.0f, 0.0f};
    if (lane < n) st = *reinterpret_cast<const f32x4*>(ml + lane * ml_stride);
    float src[kFew][kPer];
#pragma unroll
    for (int i = 0; i < kFew; ++i)
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        src[i][k] = i < n ? po[(int64_t)i * po_stride + kPer * lane + k] : 0.0f;
    const float mx = wave_max(st[0]);
    const float wgt = lane < n ? fast_exp2(st[0] - mx) : 0.0f;
    float acc[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) acc[k] = 0.0f;
#pragma unroll
    for (int i = 0; i < kFew; ++i) {
      if (i >= n) break;
      const float wi = __shfl(wgt, i, 64);
#pragma unroll
      for (int k = 0; k < kPer; ++k) acc[k] += wi * src[i][k];
    }
    const float inv = 1.0f / wave_sum(wgt * st[1]);
    if (kPer == 2) {
      *reinterpret_cast<uint32_t*>(orow + 2 * lane) = pack_bf16x2(acc[0] * inv, acc[kPer - 1] * inv);
    } else {
      const uint32_t w = pack_bf16x2(acc[0] * inv, 0.0f);
      orow[lane] = (uint16_t)(w & 0xFFFFu);
    }
    if (lse_out) {
      const float l_ex = wave_sum(wgt * st[2]);
      if (lane == 0) *lse_out = (mx + __log2f(l_ex)) * kLn2;
    }
    return;
  }
  float mx = kNoMax;
  for (int s = lane; s < n; s += 64) mx = fmaxf(mx, ml[s * ml_stride]);
  mx = wave_max(mx);

  float acc[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) acc[i] = 0.0f;
  float l_round = 0.0f, l_ex = 0.0f;
  for (int s0 = 0; s0 < n; s0 += 64) {
    const int s = s0 + lane;
    float wgt = 0.0f;
    if (s < n) {
      const f32x4 st = *reinterpret_cast<const f32x4*>(ml + s * ml_stride);
      wgt = fast_exp2(st[0] - mx);
      l_round += wgt * st[1];
      l_ex += wgt * st[2];
    }
    const int cnt = min(64, n - s0);
    // kFew partials at a time, all loaded before they are summed (in split order)
    for (int i0 = 0; i0 < cnt; i0 += kFew) {
      float src[kFew][kPer];
#pragma unroll
      for (int i = 0; i < kFew; ++i)
#pragma unroll
        for (int k = 0; k < kPer; ++k)
          src[i][k] = i0 + i < cnt ? po[(int64_t)(s0 + i0 + i) * po_stride + kPer * lane + k]
                                   : 0.0f;
#pragma unroll
      for (int i = 0; i < kFew; ++i) {
        if (i0 + i >= cnt) break;
        const float wi = __shfl(wgt, i0 + i, 64);
#pragma unroll
        for (int k = 0; k < kPer; ++k) acc[k] += wi * src[i][k];
      }
    }
  }
  l_round = wave_sum(l_round);
  const float inv = 1.0f / l_round;
  if (kPer == 2) {
    *reinterpret_cast<uint32_t*>(orow + 2 * lane) = pack_bf16x2(acc[0] * inv, acc[kPer - 1] * inv);
  } else {
    const uint32_t w = pack_bf16x2(acc[0] * inv, 0.0f);
    orow[lane] = (uint16_t)(w & 0xFFFFu);
  }
  if (lse_out) {
    l_ex = wave_sum(l_ex);
    if (lane == 0) *lse_out = (mx + __log2f(l_ex)) * kLn2;
  }
}

// v_mfma_f32_32x32x16_bf16.  Lane layouts (checked on gfx950):
//   A: lane l holds row l%32, k = 8*(l/32) .. +7;  B: lane l holds column l%32, same k;
//   D: lane l register r holds row 8*(r/4) + 4*(l/32) + r%4, column l%32.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16.  A: lane l row l%16, k = 8*(l/16) .. +7; B: column l%16;
//   D: lane l register r holds row 4*(l/16) + r, column l%16.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Row permutation for the 32x32 tiles.  When the 32 rows of an S^T = K.Q^T tile are the
// keys kappa(0..31), the D registers r = 0..7 of lane l hold keys 8*(l/32) + r and
// registers 8..15 hold 16 + 8*(l/32) + (r - 8): each lane owns runs of 8 consecutive
// keys, which is exactly the B operand of the P.V product over 16 keys.  The V^T operand
// of that product is read so that its rows follow the same pattern over the head-dim
// entries, which makes each lane's outputs 8 consecutive entries (16-byte stores).
__device__ __forceinline__ int perm32(int rho) {
  const int j = rho >> 3, h = (rho >> 2) & 1, r = rho & 3;
  return 16 * (j >> 1) + 8 * h + 4 * (j & 1) + r;
}

}  // namespace tide
