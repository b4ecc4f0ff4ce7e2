/* Exercises the oracle's C entry points (oracle/oracle.c) on random small shapes and on
 * its error paths, so that a sanitizer build (test_sanitizers.py: gcc with
 * -fsanitize=address,undefined) checks every access they make.  No results are
 * compared here; the oracle's values are pinned by test_oracle.py.  Exits 0 when every
 * call returned the status it should. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                     uint16_t* v_pool, int64_t num_pages, const int32_t* bt, int32_t bt_stride,
                     int32_t num_tasks, const int32_t* prefix_lens, const int32_t* extend_lens,
                     int32_t hkv, int32_t d);
int oracle_attention(const uint16_t* q_sel, int64_t n_sel, const int64_t* sel_rows,
                     const uint16_t* k_pool, const uint16_t* v_pool, int64_t num_pages,
                     const int32_t* bt, int32_t bt_stride, int32_t num_tasks,
                     const int32_t* prefix_lens, const int32_t* extend_lens, int32_t hq,
                     int32_t hkv, int32_t d, double scale, double* out, double* lse,
                     int32_t nthreads);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next(void) {  /* xorshift64* */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int pick(int n) { return (int)(next() % (uint32_t)n); }
/* a random finite bf16 of moderate size */
static uint16_t bf16(void) { return (uint16_t)(0x3C00 + pick(0x0600)) | (uint16_t)(pick(2) << 15); }

static int one_case(int trial) {
  const int hkv = 1 + pick(4), g = 1 + pick(4), hq = hkv * g, d = pick(2) ? 64 : 128;
  const int n = 1 + pick(4);
  int32_t pl[4], el[4], pages_of[4];
  int total_pages = 0, rows = 0;
  for (int b = 0; b < n; ++b) {
    pl[b] = pick(70);
    el[b] = pick(40);
    pages_of[b] = (pl[b] + el[b] + 15) / 16;
    total_pages += pages_of[b];
    rows += el[b];
  }
  const int stride = 8;
  int32_t* bt = calloc((size_t)n * stride, sizeof(int32_t));
  int next_page = 0;
  for (int b = 0; b < n; ++b)
    for (int i = 0; i < stride; ++i) bt[b * stride + i] = i < pages_of[b] ? next_page++ : -1;
  const size_t pool = (size_t)(total_pages > 0 ? total_pages : 1) * hkv * 16 * d;
  uint16_t* kp = malloc(pool * 2);
  uint16_t* vp = malloc(pool * 2);
  for (size_t i = 0; i < pool; ++i) kp[i] = bf16(), vp[i] = bf16();
  const size_t nk = (size_t)(rows > 0 ? rows : 1) * hkv * d;
  uint16_t* kn = malloc(nk * 2);
  uint16_t* vn = malloc(nk * 2);
  for (size_t i = 0; i < nk; ++i) kn[i] = bf16(), vn[i] = bf16();
  int bad = 0;
  int rc = oracle_kv_append(kn, vn, kp, vp, total_pages > 0 ? total_pages : 1, bt, stride, n, pl,
                            el, hkv, d);
  if (rc != 0) bad |= 1, printf("trial %d: append rc %d\n", trial, rc);
  if (rows > 0) {
    const int nsel = 1 + pick(rows);
    int64_t* sel = malloc(sizeof(int64_t) * nsel);
    for (int i = 0; i < nsel; ++i) sel[i] = pick(rows);
    uint16_t* q = malloc((size_t)nsel * hq * d * 2);
    for (size_t i = 0; i < (size_t)nsel * hq * d; ++i) q[i] = bf16();
    double* out = malloc(sizeof(double) * nsel * hq * d);
    double* lse = malloc(sizeof(double) * nsel * hq);
    rc = oracle_attention(q, nsel, sel, kp, vp, total_pages, bt, stride, n, pl, el, hq, hkv, d,
                          0.125, out, lse, 1 + pick(3));
    if (rc != 0) bad |= 1, printf("trial %d: attention rc %d\n", trial, rc);
    /* a row index past the packed rows is refused */
    sel[0] = rows;
    if (oracle_attention(q, 1, sel, kp, vp, total_pages, bt, stride, n, pl, el, hq, hkv, d,
                         0.125, out, lse, 1) == 0)
      bad |= 1, printf("trial %d: bad row accepted\n", trial);
    /* a block-table entry out of range is refused, not dereferenced */
    int b = 0;
    while (b < n && el[b] == 0) ++b;
    if (b < n) {
      const int32_t keep = bt[b * stride];
      bt[b * stride] = total_pages + 3;
      sel[0] = 0;
      for (int t = 0; t < b; ++t) sel[0] += el[t];
      if (oracle_attention(q, 1, sel, kp, vp, total_pages, bt, stride, n, pl, el, hq, hkv, d,
                           0.125, out, lse, 1) != -3)
        bad |= 1, printf("trial %d: bad page accepted\n", trial);
      bt[b * stride] = keep;
      /* append writes only the pages of positions pl[b] .. pl[b] + el[b] - 1 */
      const int lp = pl[b] / 16;
      const int32_t keep2 = bt[b * stride + lp];
      bt[b * stride + lp] = -1;
      if (oracle_kv_append(kn, vn, kp, vp, total_pages, bt, stride, n, pl, el, hkv, d) != -3)
        bad |= 1, printf("trial %d: bad page accepted by append\n", trial);
      bt[b * stride + lp] = keep2;
    }
    free(sel), free(q), free(out), free(lse);
  }
  free(bt), free(kp), free(vp), free(kn), free(vn);
  return bad;
}

int main(void) {
  int bad = 0;
  for (int t = 0; t < 300; ++t) bad |= one_case(t);
  printf(bad ? "FAIL\n" : "ok\n");
  return bad;
}
