/*
 * oracle.c -- plain, slow fp64 CPU reference for the paged-KV resume-attention path.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
 * baseline call this code; the library's compute path never does.  It shares no
 * code, header or table with the HIP kernels.
 *
 * What it computes (TideRL, arXiv 2608.10402):
 *   A resumed multi-turn task keeps its KV cache (Continuous Task Batching, Section 4;
 *   resume with cache locality, Section 4.2) and only attends the new tokens against
 *   the retained prefix; an evicted cache forces a recompute of the whole history
 *   (challenge C1, Section 2.2), as does a weight update (Section 5.2, cache-free task
 *   migration).  Both must give the same continuation, which is why a hit is pure
 *   savings.  The attention is ordinary scaled dot-product attention (Vaswani et al.
 *   2017; the paper relies on it without restating it):
 *       s_p = scale * sum_i q_i k_{p,i},  p = 0 .. t   (t = the query's own position)
 *       m = max_p s_p,  w_p = exp(s_p - m),  Z = sum_p w_p
 *       o = sum_p w_p v_p / Z,  lse = m + log Z
 *   with the KV head of query head h being floor(h / (Hq / Hkv)).
 *
 * Storage follows the library's documented pool layout, reimplemented here from
 * that description:
 *   K pool and V pool  [num_pages][Hkv][16][d]  (token slots, then head-dim contiguous)
 *   position p of task b lives in page block_table[b][p / 16], slot p % 16.
 * Values are bf16 bit patterns; every one converts to fp64 exactly.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_PAGE 16

static double bf16_bits_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Element i of the row at (page, kv head g, slot) in either pool. */
static size_t slot_index(int64_t page, int g, int slot, int i, int hkv, int d) {
  return (((size_t)page * (size_t)hkv + (size_t)g) * ORACLE_PAGE + (size_t)slot) * (size_t)d +
         (size_t)i;
}

/* Physical page of logical position p of task b, or -1 if the table does not map it. */
static int64_t page_of(const int32_t* bt, int32_t bt_stride, int64_t num_pages, int b, int64_t p) {
  int64_t lp = p / ORACLE_PAGE;
  if (lp >= bt_stride) return -1;
  int64_t page = bt[(size_t)b * (size_t)bt_stride + (size_t)lp];
  if (page < 0 || page >= num_pages) return -1;
  return page;
}

/*
 * Append: copy the K/V rows of each task's new tokens into the pool image.
 * New token j of task b is position prefix_lens[b] + j and row indptr_b + j of
 * k_new / v_new ([rows][Hkv][d]).  Returns 0, or -3 when a position has no valid page.
 */
int oracle_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                     uint16_t* v_pool, int64_t num_pages, const int32_t* bt, int32_t bt_stride,
                     int32_t num_tasks, const int32_t* prefix_lens, const int32_t* extend_lens,
                     int32_t hkv, int32_t d) {
  int64_t row = 0;
  for (int b = 0; b < num_tasks; ++b) {
    for (int32_t j = 0; j < extend_lens[b]; ++j, ++row) {
      int64_t pos = (int64_t)prefix_lens[b] + j;
      int64_t page = page_of(bt, bt_stride, num_pages, b, pos);
      if (page < 0) return -3;
      int slot = (int)(pos % ORACLE_PAGE);
      for (int g = 0; g < hkv; ++g) {
        for (int i = 0; i < d; ++i) {
          size_t src = ((size_t)row * (size_t)hkv + (size_t)g) * (size_t)d + (size_t)i;
          k_pool[slot_index(page, g, slot, i, hkv, d)] = k_new[src];
          v_pool[slot_index(page, g, slot, i, hkv, d)] = v_new[src];
        }
      }
    }
  }
  return 0;
}

/*
 * Attention for a selection of query rows.
 *   q_sel     bf16 [n_sel][Hq][d]: the query rows themselves
 *   sel_rows  int64 [n_sel]: the packed row index of each (row r belongs to task b when
 *             indptr_b <= r < indptr_{b+1}, indptr = prefix sums of extend_lens)
 *   out       fp64 [n_sel][Hq][d];  lse  fp64 [n_sel][Hq]
 * Row j of task b is at position t = prefix_lens[b] + j and attends to keys 0 .. t.
 * Returns 0, -1 on a bad row index, -3 when a needed position has no valid page.
 */
int oracle_attention(const uint16_t* q_sel, int64_t n_sel, const int64_t* sel_rows,
                     const uint16_t* k_pool, const uint16_t* v_pool, int64_t num_pages,
                     const int32_t* bt, int32_t bt_stride, int32_t num_tasks,
                     const int32_t* prefix_lens, const int32_t* extend_lens, int32_t hq,
                     int32_t hkv, int32_t d, double scale, double* out, double* lse,
                     int32_t nthreads) {
  int64_t* indptr = (int64_t*)malloc(sizeof(int64_t) * ((size_t)num_tasks + 1));
  if (!indptr) return -2;
  indptr[0] = 0;
  for (int b = 0; b < num_tasks; ++b) indptr[b + 1] = indptr[b] + extend_lens[b];
  const int group = hq / hkv;
  int status = 0;

#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
  for (int64_t item = 0; item < n_sel * (int64_t)hq; ++item) {
    int64_t sel = item / hq;
    int h = (int)(item % hq);
    int64_t row = sel_rows[sel];
    if (row < 0 || row >= indptr[num_tasks]) {
#pragma omp atomic write
      status = -1;
      continue;
    }
    int b = 0;
    while (indptr[b + 1] <= row) ++b;
    int64_t t = (int64_t)prefix_lens[b] + (row - indptr[b]);
    int g = h / group;

    double* q = (double*)malloc(sizeof(double) * (size_t)d);
    double* s = (double*)malloc(sizeof(double) * (size_t)(t + 1));
    double* o = out + ((size_t)sel * (size_t)hq + (size_t)h) * (size_t)d;
    for (int i = 0; i < d; ++i)
      q[i] = bf16_bits_to_double(q_sel[((size_t)sel * (size_t)hq + (size_t)h) * (size_t)d + i]);

    /* scores over every key the row may see */
    int bad = 0;
    for (int64_t p = 0; p <= t; ++p) {
      int64_t page = page_of(bt, bt_stride, num_pages, b, p);
      if (page < 0) {
        bad = 1;
        break;
      }
      int slot = (int)(p % ORACLE_PAGE);
      double dot = 0.0;
      for (int i = 0; i < d; ++i)
        dot += q[i] * bf16_bits_to_double(k_pool[slot_index(page, g, slot, i, hkv, d)]);
      s[p] = scale * dot;
    }
    if (bad) {
#pragma omp atomic write
      status = -3;
      free(q);
      free(s);
      continue;
    }

    /* softmax */
    double m = s[0];
    for (int64_t p = 1; p <= t; ++p)
      if (s[p] > m) m = s[p];
    double z = 0.0;
    for (int64_t p = 0; p <= t; ++p) {
      s[p] = exp(s[p] - m);
      z += s[p];
    }

    /* weighted sum of values */
    for (int i = 0; i < d; ++i) o[i] = 0.0;
    for (int64_t p = 0; p <= t; ++p) {
      int64_t page = page_of(bt, bt_stride, num_pages, b, p);
      int slot = (int)(p % ORACLE_PAGE);
      for (int i = 0; i < d; ++i)
        o[i] += s[p] * bf16_bits_to_double(v_pool[slot_index(page, g, slot, i, hkv, d)]);
    }
    for (int i = 0; i < d; ++i) o[i] /= z;
    lse[(size_t)sel * (size_t)hq + (size_t)h] = m + log(z);
    free(q);
    free(s);
  }
  free(indptr);
  return status;
}
