/*
 * Counter-based normal generator for the synthetic workloads.
 *
 * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as
 * 1, 2, 3", SC'11) maps a 128-bit counter and a 64-bit key to four uniformly
 * distributed 32-bit words.  Element e of a stream takes counter block e/4:
 *     ctr = {lo32(e/4), hi32(e/4), stream_a, stream_b},  key = {lo32(seed), hi32(seed)}
 * and the four words become four N(0,1) samples by the Box-Muller transform
 * (pairs (w0,w1) and (w2,w3); uniforms u = (w >> 8) * 2^-24 + 2^-25 in (0,1], in fp32),
 * each rounded to bf16 with round-to-nearest-even.  Every element can be produced
 * on its own, so any slice of a tensor (one task, a range of token rows) is
 * generated without producing the rest.
 *
 * This file is input generation only: it contains none of the attention arithmetic.
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox_round(uint32_t c[4], const uint32_t k[2]) {
  uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
  uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
  uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  uint32_t n0 = hi1 ^ c[1] ^ k[0];
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

/* Philox4x32 with 10 rounds; the key is bumped by the Weyl constants between rounds. */
void tg_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k[0] += PHILOX_W0;
      k[1] += PHILOX_W1;
    }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof(c));
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t rounding = 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)((u + rounding) >> 16);
}

static inline float unit_open(uint32_t w) {
  return (float)(w >> 8) * (1.0f / 16777216.0f) + (1.0f / 33554432.0f);
}

static void normals_of_block(uint64_t blk, uint32_t sa, uint32_t sb, const uint32_t key[2],
                             float z[4]) {
  uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), sa, sb};
  uint32_t w[4];
  tg_philox4x32_10(ctr, key, w);
  const float two_pi = 6.2831853071795865f;
  for (int pair = 0; pair < 2; ++pair) {
    float u1 = unit_open(w[2 * pair]);
    float u2 = unit_open(w[2 * pair + 1]);
    float r = sqrtf(-2.0f * logf(u1));
    float s, c;
    sincosf(two_pi * u2, &s, &c);
    z[2 * pair] = r * c;
    z[2 * pair + 1] = r * s;
  }
}

/* out[i] = bf16(N(0,1) sample for element first+i of stream (seed, sa, sb)), i in [0, n). */
void tg_normal_bf16(uint64_t seed, uint32_t sa, uint32_t sb, uint64_t first, int64_t n,
                    uint16_t* out, int nthreads) {
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  if (n <= 0) return;
  uint64_t blk_lo = first >> 2;
  uint64_t blk_hi = (first + (uint64_t)n - 1) >> 2;
  int64_t nblk = (int64_t)(blk_hi - blk_lo + 1);
#pragma omp parallel for schedule(static) num_threads(nthreads) if (nblk > 4096)
  for (int64_t bi = 0; bi < nblk; ++bi) {
    uint64_t blk = blk_lo + (uint64_t)bi;
    float z[4];
    normals_of_block(blk, sa, sb, key, z);
    for (int j = 0; j < 4; ++j) {
      uint64_t e = blk * 4 + (uint64_t)j;
      if (e < first || e >= first + (uint64_t)n) continue;
      out[e - first] = f32_to_bf16_rne(z[j]);
    }
  }
}

/* Same as tg_normal_bf16 but writes fp32 samples (used to test the distribution). */
void tg_normal_f32(uint64_t seed, uint32_t sa, uint32_t sb, uint64_t first, int64_t n,
                   float* out, int nthreads) {
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  if (n <= 0) return;
  uint64_t blk_lo = first >> 2;
  uint64_t blk_hi = (first + (uint64_t)n - 1) >> 2;
  int64_t nblk = (int64_t)(blk_hi - blk_lo + 1);
#pragma omp parallel for schedule(static) num_threads(nthreads) if (nblk > 4096)
  for (int64_t bi = 0; bi < nblk; ++bi) {
    uint64_t blk = blk_lo + (uint64_t)bi;
    float z[4];
    normals_of_block(blk, sa, sb, key, z);
    for (int j = 0; j < 4; ++j) {
      uint64_t e = blk * 4 + (uint64_t)j;
      if (e < first || e >= first + (uint64_t)n) continue;
      out[e - first] = z[j];
    }
  }
}

/* Several slices of one tensor family at once: segment i is samples
   first[i] .. first[i]+len[i]-1 of stream (sa, sb[i]); the segments are written one after
   another into out.  Used to fetch rows of many tasks in one call. */
void tg_normal_bf16_segments(uint64_t seed, uint32_t sa, int64_t nseg, const uint32_t* sb,
                             const uint64_t* first, const int64_t* len, uint16_t* out,
                             int nthreads) {
  if (nseg <= 0) return;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nseg + 1));
  if (!off) return;
  off[0] = 0;
  for (int64_t i = 0; i < nseg; ++i) off[i + 1] = off[i] + len[i];
#pragma omp parallel for schedule(dynamic, 16) num_threads(nthreads) if (off[nseg] > 65536)
  for (int64_t i = 0; i < nseg; ++i)
    tg_normal_bf16(seed, sa, sb[i], first[i], len[i], out + off[i], 1);
  free(off);
}
