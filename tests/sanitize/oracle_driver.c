/* Runs every entry point of the C oracle (jf_oracle.c) on small random
 * inputs, including ragged lengths, partial pages, invalid page IDs and
 * rejected arguments, in a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer.  Exits non-zero on the first failed check; the
 * sanitizers abort on their own findings.  Test infrastructure only. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "jf_oracle.h"

static int g_checks = 0;
#define CHECK(c)                                                          \
  do {                                                                    \
    ++g_checks;                                                           \
    if (!(c)) {                                                           \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
      exit(1);                                                            \
    }                                                                     \
  } while (0)

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64(void) { /* splitmix64 */
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static double uniform(void) { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }

/* fp16 bits of a value drawn from [-4, 4), with an occasional outlier. */
static uint16_t rand_half(void) {
  double x = 8.0 * uniform() - 4.0;
  if ((next_u64() & 63) == 0) x *= 300.0;
  return jfo_double_to_half(x, 0);
}

static void fill_half(uint16_t* p, size_t n) {
  for (size_t i = 0; i < n; ++i) p[i] = rand_half();
}

static void* xcalloc(size_t n, size_t s) {
  void* p = calloc(n ? n : 1, s);
  CHECK(p != NULL);
  return p;
}

static void halves(void) {
  /* round-trips and directed roundings of a few values */
  const double vals[] = {0.0, 1.0, -2.5, 65504.0, 6.103515625e-05, 5.960464477539063e-08, 1e-9};
  for (size_t i = 0; i < sizeof vals / sizeof vals[0]; ++i) {
    const uint16_t h = jfo_double_to_half(vals[i], 0);
    CHECK(jfo_half_to_double(h) == vals[i] || vals[i] == 1e-9);
    CHECK(jfo_half_to_double(jfo_double_to_half(vals[i], 1)) <= vals[i]);
    CHECK(jfo_half_to_double(jfo_double_to_half(vals[i], 2)) >= vals[i]);
    CHECK(jfo_float_to_half((float)vals[i], 0) == h);
  }
  CHECK(isinf(jfo_half_to_double(jfo_double_to_half(1e6, 0))));
  for (int i = 0; i < 100000; ++i) {
    const uint16_t h = (uint16_t)next_u64();
    const double x = jfo_half_to_double(h);
    if (!isnan(x)) CHECK(jfo_double_to_half(x, 0) == h || x == 0.0);
  }
}

static void groups(void) {
  const int32_t Gs[] = {16, 32, 64, 128};
  for (int gi = 0; gi < 4; ++gi) {
    const int32_t G = Gs[gi];
    const int64_t n = 257;
    uint16_t* x = xcalloc((size_t)n * G, 2);
    uint8_t* codes = xcalloc((size_t)n * G, 1);
    uint16_t* s = xcalloc((size_t)n, 2);
    uint16_t* b = xcalloc((size_t)n, 2);
    fill_half(x, (size_t)n * G);
    for (int32_t j = 0; j < G; ++j) x[j] = x[0]; /* a constant group */
    jfo_quantize_groups(x, n, G, codes, s, b);
    for (int64_t i = 0; i < n * G; ++i) CHECK(codes[i] < 16);
    free(x), free(codes), free(s), free(b);
  }
}

/* A pool, a few ragged requests appended in two steps, then decode, prefill
 * and reconstruction over it. */
static void pool_paths(int32_t P, int32_t Hkv, int32_t d, int32_t G, int32_t Hq) {
  const int32_t NP = 24, B = 3, max_pages = 8;
  const jfo_layout L = {P, Hkv, d, G, NP};
  const size_t cbytes = jfo_codes_bytes(&L), melems = jfo_meta_elems(&L);
  uint8_t* kc = xcalloc(cbytes, 1);
  uint8_t* vc = xcalloc(cbytes, 1);
  uint16_t* km = xcalloc(melems, 2);
  uint16_t* vm = xcalloc(melems, 2);
  int32_t tables[3 * 8];
  int32_t next = NP - 1; /* pages handed out in reverse order */
  for (int i = 0; i < B * max_pages; ++i) tables[i] = -1;
  const int32_t lens[3] = {1, P * 2 + 3, P * 5};
  for (int32_t b = 0; b < B; ++b)
    for (int32_t j = 0; j * P < lens[b]; ++j) tables[b * max_pages + j] = next--;
  /* append in two steps: the first row of each request, then the rest */
  int32_t cu[4] = {0}, start[3];
  for (int step = 0; step < 2; ++step) {
    int32_t tot = 0;
    for (int32_t b = 0; b < B; ++b) {
      start[b] = step ? 1 : 0;
      const int32_t n = step ? lens[b] - 1 : 1;
      cu[b] = tot;
      tot += n;
    }
    cu[B] = tot;
    uint16_t* kn = xcalloc((size_t)tot * Hkv * d, 2);
    uint16_t* vn = xcalloc((size_t)tot * Hkv * d, 2);
    fill_half(kn, (size_t)tot * Hkv * d);
    fill_half(vn, (size_t)tot * Hkv * d);
    CHECK(jfo_quantize_append(&L, kc, km, vc, vm, kn, vn, cu, start, tables, B, max_pages) == 0);
    free(kn), free(vn);
  }
  { /* an append through a page ID outside the pool is refused */
    int32_t bad[8];
    for (int i = 0; i < 8; ++i) bad[i] = NP + i;
    int32_t c1[2] = {0, 1}, s1[1] = {0};
    uint16_t row[2 * 128 * 8];
    memset(row, 0, sizeof row);
    CHECK(jfo_quantize_append(&L, kc, km, vc, vm, row, row, c1, s1, bad, 1, 8) == -1);
  }
  double* vec = xcalloc((size_t)d, sizeof(double));
  jfo_dequant_vector(&L, kc, km, 0, tables[max_pages], 0, 1, vec);
  jfo_dequant_vector(&L, vc, vm, 1, tables[max_pages], Hkv - 1, P - 1, vec);
  for (int32_t i = 0; i < d; ++i) CHECK(isfinite(vec[i]));
  free(vec);

  /* decode */
  uint16_t* q = xcalloc((size_t)B * Hq * d, 2);
  for (size_t i = 0; i < (size_t)B * Hq * d; ++i) q[i] = jfo_double_to_half(uniform() - 0.5, 0);
  double* out = xcalloc((size_t)B * Hq * d, sizeof(double));
  const double alpha = 1.0 / sqrt((double)d);
  CHECK(jfo_decode(&L, kc, km, vc, vm, q, B, Hq, tables, max_pages, lens, alpha, out) == 0);
  for (size_t i = 0; i < (size_t)B * Hq * d; ++i) CHECK(isfinite(out[i]));
  if (Hkv > 1) /* query heads not a multiple of the KV heads */
    CHECK(jfo_decode(&L, kc, km, vc, vm, q, B, Hq + 1, tables, max_pages, lens, alpha, out) == -1);
  const int32_t too_long[3] = {1, P * max_pages + 1, 2};
  CHECK(jfo_decode(&L, kc, km, vc, vm, q, B, Hq, tables, max_pages, too_long, alpha, out) == -1);

  /* prefill of a 5-row chunk after request 1's prefix, all rows and a subset */
  const int32_t T = 5, prefix = lens[1];
  int32_t ptab[8];
  for (int i = 0; i < 8; ++i) ptab[i] = tables[max_pages + i];
  uint16_t* pq = xcalloc((size_t)T * Hq * d, 2);
  uint16_t* pk = xcalloc((size_t)T * Hkv * d, 2);
  uint16_t* pv = xcalloc((size_t)T * Hkv * d, 2);
  fill_half(pk, (size_t)T * Hkv * d);
  fill_half(pv, (size_t)T * Hkv * d);
  for (size_t i = 0; i < (size_t)T * Hq * d; ++i) pq[i] = jfo_double_to_half(uniform() - 0.5, 0);
  double* pout = xcalloc((size_t)T * Hq * d, sizeof(double));
  for (int cq = 0; cq < 2; ++cq)
    CHECK(jfo_prefill(&L, kc, km, vc, vm, pq, pk, pv, T, Hq, ptab, max_pages, prefix, alpha, cq,
                      NULL, T, pout) == 0);
  const int32_t rows[2] = {4, 0};
  CHECK(jfo_prefill(&L, kc, km, vc, vm, pq, pk, pv, T, Hq, ptab, max_pages, prefix, alpha, 1, rows,
                    2, pout) == 0);
  CHECK(jfo_prefill(&L, kc, km, vc, vm, pq, pk, pv, T, Hq, ptab, max_pages, 0, alpha, 0, NULL, T,
                    pout) == 0);
  for (size_t i = 0; i < (size_t)T * Hq * d; ++i) CHECK(isfinite(pout[i]));

  /* reconstruction of both K and V, including a page outside the pool */
  const int32_t n = lens[2];
  uint16_t* rec = xcalloc((size_t)Hkv * n * d, 2);
  int32_t rtab[8];
  for (int i = 0; i < 8; ++i) rtab[i] = tables[2 * max_pages + i];
  rtab[1] = -1;
  CHECK(jfo_reconstruct(&L, kc, km, 0, rtab, max_pages, n, 0, Hkv, rec) == 0);
  for (int32_t g = 0; g < Hkv; ++g)
    for (int32_t t = P; t < 2 * P; ++t)
      for (int32_t i = 0; i < d; ++i) CHECK(rec[((size_t)g * n + t) * d + i] == 0);
  CHECK(jfo_reconstruct(&L, vc, vm, 1, rtab, max_pages, n, Hkv - 1, 1, rec) == 0);
  CHECK(jfo_reconstruct(&L, vc, vm, 1, rtab, max_pages, n, Hkv - 1, 2, rec) == -1);
  CHECK(jfo_reconstruct(&L, vc, vm, 1, rtab, max_pages, P * max_pages + 1, 0, 1, rec) == -1);

  free(q), free(out), free(pq), free(pk), free(pv), free(pout), free(rec);
  free(kc), free(vc), free(km), free(vm);
}

int main(void) {
  halves();
  groups();
  pool_paths(16, 2, 64, 32, 4);
  pool_paths(32, 1, 128, 64, 3);
  pool_paths(16, 4, 128, 128, 8);
  printf("oracle driver: %d checks passed\n", g_checks);
  return 0;
}
