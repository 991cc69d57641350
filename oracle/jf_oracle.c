/*
 * jf_oracle.c -- plain, slow, obviously-correct CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY (see jf_oracle.h): used by the tests, the smoke
 * check and the benchmark's CPU baseline, never by the product path.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -fPIC
 *        -shared jf_oracle.c -o libjforacle.so -lm
 * (-ffp-contract=off keeps every binary32 operation of the quantizer a
 * separately rounded IEEE operation, which is what the encoding specifies.)
 */
#include "jf_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int jfo_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void jfo_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------
 * binary16 from its definition: sign, 5-bit biased exponent, 10-bit
 * fraction; exponent 0 holds subnormals (fraction * 2^-24).
 * ---------------------------------------------------------------------- */
double jfo_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)m, -24);
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = ldexp((double)(m | 0x400), e - 25);
  return sign ? -v : v;
}

/* Largest non-negative binary16 pattern (0..0x7bff) whose value is <= a,
 * for finite a >= 0.  Positive binary16 patterns are ordered like their
 * values, so a bisection over the patterns finds it. */
static uint16_t half_floor_pattern(double a) {
  uint16_t lo = 0, hi = 0x7bff; /* value(lo) <= a is invariant */
  if (jfo_half_to_double(hi) <= a) return hi;
  while (hi - lo > 1) {
    uint16_t mid = (uint16_t)((lo + hi) / 2);
    if (jfo_half_to_double(mid) <= a)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

/* Round the binary64 value x to binary16.  Candidates are the two
 * neighbours of |x|; "away" is the larger magnitude.  Beyond the largest
 * finite value the upper neighbour is infinity, which round-to-nearest
 * reaches from 65520 up (the halfway point to 2^16, where the next binade
 * would start).  The distances to the neighbours are exact: the neighbours
 * and every binary64 value in their range are dyadic with few enough bits. */
uint16_t jfo_double_to_half(double x, int mode) {
  if (isnan(x)) return 0x7e00;
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (isinf(x)) {
    if (mode == 1 && !sign) return 0x7bff; /* +inf toward -inf: max finite */
    if (mode == 2 && sign) return 0xfbff;  /* -inf toward +inf             */
    return (uint16_t)(sign | 0x7c00);
  }
  uint16_t lo = half_floor_pattern(a);
  double vlo = jfo_half_to_double(lo);
  if (vlo == a) return (uint16_t)(sign | lo);
  uint16_t up = (uint16_t)(lo + 1); /* 0x7c00 (inf) when lo is the max */
  double vup = (up == 0x7c00) ? 65536.0 : jfo_half_to_double(up);
  uint16_t mag;
  if (mode == 0) {
    double dlo = a - vlo, dup = vup - a; /* exact: a and both ends are dyadic */
    if (dlo < dup)
      mag = lo;
    else if (dup < dlo)
      mag = up;
    else
      mag = (lo & 1) ? up : lo; /* tie: even last fraction bit */
  } else {
    /* toward -inf: magnitude down for +, up for -; toward +inf: reverse */
    int mag_up = (mode == 1) ? (sign != 0) : (sign == 0);
    mag = mag_up ? up : lo;
  }
  return (uint16_t)(sign | mag);
}

/* binary32 input: exact in binary64, so the same rounding. */
uint16_t jfo_float_to_half(float f, int mode) { return jfo_double_to_half((double)f, mode); }

static float half_to_float(uint16_t h) { return (float)jfo_half_to_double(h); }

/* ------------------------------------------------------------------------
 * Group quantizer.  For one group x_0..x_{G-1} (fp16, finite):
 *   1. mn, mx: exact minimum and maximum in binary32 (-0 below +0).
 *   2. bias  = fp16(mn) rounded toward -inf (exact for fp16 inputs).
 *   3. range = mx - mn; step = range / 15 (binary32, round to nearest);
 *      scale = fp16(step) rounded toward +inf (+0 when range is 0).
 *   4. scale 0: every code 0.  Otherwise
 *      r_i = (x_i - bias) / scale   (two separately rounded binary32 ops),
 *      code_i = clamp(round-half-even(r_i), 0, 15).
 * Rounding the bias down and the scale up keeps [mn, mx] inside the 16
 * levels bias + k*scale, so each element is within scale/2 of its level.
 * ---------------------------------------------------------------------- */
void jfo_quantize_group(const uint16_t* x, int32_t G, uint8_t* codes,
                        uint16_t* scale, uint16_t* bias) {
  /* -0 orders below +0, so the result does not depend on element order */
  float mn = half_to_float(x[0]), mx = mn;
  for (int32_t i = 1; i < G; ++i) {
    float v = half_to_float(x[i]);
    if (v < mn || (v == mn && signbit(v) && !signbit(mn))) mn = v;
    if (v > mx || (v == mx && !signbit(v) && signbit(mx))) mx = v;
  }
  uint16_t b16 = jfo_float_to_half(mn, 1);
  volatile float range = mx - mn;
  volatile float step = range / 15.0f;
  uint16_t s16 = (range == 0.0f) ? (uint16_t)0 : jfo_float_to_half(step, 2);
  *scale = s16;
  *bias = b16;
  float sf = half_to_float(s16), bf = half_to_float(b16);
  for (int32_t i = 0; i < G; ++i) {
    if (s16 == 0) {
      codes[i] = 0;
      continue;
    }
    volatile float diff = half_to_float(x[i]) - bf;
    volatile float r = diff / sf;
    float q = rintf(r); /* default rounding mode: nearest, ties to even */
    if (q < 0.0f) q = 0.0f;
    if (q > 15.0f) q = 15.0f;
    codes[i] = (uint8_t)q;
  }
}

void jfo_quantize_groups(const uint16_t* x, int64_t n, int32_t G,
                         uint8_t* codes, uint16_t* scales, uint16_t* biases) {
  for (int64_t i = 0; i < n; ++i)
    jfo_quantize_group(x + i * G, G, codes + i * G, scales + i, biases + i);
}

/* ------------------------------------------------------------------------
 * Pool layout (jf_oracle.h).  Offsets are in bytes for codes, in fp16
 * elements for meta.
 * ---------------------------------------------------------------------- */
size_t jfo_codes_bytes(const jfo_layout* L) {
  return (size_t)L->num_pages * L->num_kv_heads * L->page_size *
         (L->head_dim / 2);
}

size_t jfo_meta_elems(const jfo_layout* L) {
  return (size_t)L->num_pages * L->num_kv_heads * L->page_size *
         (L->head_dim / L->group_size) * 2;
}

static size_t page_head_codes_base(const jfo_layout* L, int32_t page,
                                   int32_t kv) {
  return ((size_t)page * L->num_kv_heads + kv) * L->page_size *
         (L->head_dim / 2);
}

/* Byte holding the code of dimension i at (page, kv, slot). */
static size_t k_code_byte(const jfo_layout* L, int32_t page, int32_t kv,
                          int32_t slot, int32_t i) {
  return page_head_codes_base(L, page, kv) + (size_t)slot * (L->head_dim / 2) +
         (size_t)(i / 2);
}

static size_t v_code_byte(const jfo_layout* L, int32_t page, int32_t kv,
                          int32_t slot, int32_t i) {
  int32_t u = i / 4;           /* four-dimension chunk */
  int32_t within = (i % 4) / 2; /* byte of the chunk's two */
  return page_head_codes_base(L, page, kv) +
         ((size_t)(slot / 2) * (L->head_dim / 4) + u) * 4 +
         (size_t)(slot % 2) * 2 + within;
}

static size_t meta_index(const jfo_layout* L, int32_t page, int32_t kv,
                         int32_t slot, int32_t g) {
  size_t ng = (size_t)(L->head_dim / L->group_size);
  return ((((size_t)page * L->num_kv_heads + kv) * L->page_size + slot) * ng +
          g) * 2;
}

static int get_code(const jfo_layout* L, const uint8_t* codes, int is_v,
                    int32_t page, int32_t kv, int32_t slot, int32_t i) {
  size_t off = is_v ? v_code_byte(L, page, kv, slot, i)
                    : k_code_byte(L, page, kv, slot, i);
  return (i % 2) ? (codes[off] >> 4) & 0xf : codes[off] & 0xf;
}

static void put_code(const jfo_layout* L, uint8_t* codes, int is_v,
                     int32_t page, int32_t kv, int32_t slot, int32_t i,
                     int c) {
  size_t off = is_v ? v_code_byte(L, page, kv, slot, i)
                    : k_code_byte(L, page, kv, slot, i);
  if (i % 2)
    codes[off] = (uint8_t)((codes[off] & 0x0f) | (c << 4));
  else
    codes[off] = (uint8_t)((codes[off] & 0xf0) | c);
}

/* Quantize one fp16 vector (d values) into the pool at (page, kv, slot). */
static void store_vector(const jfo_layout* L, uint8_t* codes, uint16_t* meta,
                         int is_v, int32_t page, int32_t kv, int32_t slot,
                         const uint16_t* x) {
  int32_t G = L->group_size, ng = L->head_dim / G;
  uint8_t c[256];
  for (int32_t g = 0; g < ng; ++g) {
    uint16_t s16, b16;
    jfo_quantize_group(x + g * G, G, c, &s16, &b16);
    size_t mi = meta_index(L, page, kv, slot, g);
    meta[mi] = s16;
    meta[mi + 1] = b16;
    for (int32_t i = 0; i < G; ++i)
      put_code(L, codes, is_v, page, kv, slot, g * G + i, c[i]);
  }
}

int jfo_quantize_append(const jfo_layout* L, uint8_t* k_codes, uint16_t* k_meta,
                        uint8_t* v_codes, uint16_t* v_meta,
                        const uint16_t* k_new, const uint16_t* v_new,
                        const int32_t* cu_tok, const int32_t* start_pos,
                        const int32_t* block_tables, int32_t B,
                        int32_t max_pages) {
  int32_t d = L->head_dim, H = L->num_kv_heads, P = L->page_size;
  if (L->group_size > 256 || d % L->group_size || d % 4 || P % 2) return -1;
  for (int32_t b = 0; b < B; ++b) {
    for (int32_t r = cu_tok[b]; r < cu_tok[b + 1]; ++r) {
      int32_t pos = start_pos[b] + (r - cu_tok[b]);
      int32_t lp = pos / P;
      if (pos < 0 || lp >= max_pages) return -1;
      int32_t page = block_tables[(size_t)b * max_pages + lp];
      if (page < 0 || page >= L->num_pages) return -1;
      int32_t slot = pos % P;
      for (int32_t kv = 0; kv < H; ++kv) {
        const size_t row = ((size_t)r * H + kv) * d;
        store_vector(L, k_codes, k_meta, 0, page, kv, slot, k_new + row);
        store_vector(L, v_codes, v_meta, 1, page, kv, slot, v_new + row);
      }
    }
  }
  return 0;
}

/* x^ = scale * code + bias, in binary64. */
void jfo_dequant_vector(const jfo_layout* L, const uint8_t* codes,
                        const uint16_t* meta, int is_v, int32_t page,
                        int32_t kv, int32_t slot, double* out) {
  int32_t G = L->group_size;
  for (int32_t i = 0; i < L->head_dim; ++i) {
    size_t mi = meta_index(L, page, kv, slot, i / G);
    double s = jfo_half_to_double(meta[mi]);
    double b = jfo_half_to_double(meta[mi + 1]);
    out[i] = s * (double)get_code(L, codes, is_v, page, kv, slot, i) + b;
  }
}

/* ------------------------------------------------------------------------
 * Page -> operand reconstruction of one head group (Background, "Stored
 * format is not execution format", eq. layerbytes; Sec. 3.1, eq.
 * groupattention): the dequantized vectors of KV heads kv0 .. kv0 + g - 1 at
 * logical positions 0 .. n - 1 (page table[t / P], slot t % P), each element
 * the exact value s * q + b rounded once to binary16 (nearest, ties to even),
 * written as out[(kv - kv0) * n + t][d].  A page ID outside [0, num_pages)
 * gives zeros.
 * ---------------------------------------------------------------------- */
int jfo_reconstruct(const jfo_layout* L, const uint8_t* codes, const uint16_t* meta, int is_v,
                    const int32_t* table, int32_t max_pages, int32_t n, int32_t kv0, int32_t g,
                    uint16_t* out) {
  int32_t d = L->head_dim, P = L->page_size;
  if (d <= 0 || d > 512 || n < 0 || kv0 < 0 || g <= 0 || kv0 + g > L->num_kv_heads ||
      (int64_t)n > (int64_t)max_pages * P)
    return -1;
  double x[512];
  for (int32_t j = 0; j < g; ++j)
    for (int32_t t = 0; t < n; ++t) {
      uint16_t* o = out + ((size_t)j * n + t) * d;
      int32_t page = table[t / P];
      if (page < 0 || page >= L->num_pages) {
        for (int32_t i = 0; i < d; ++i) o[i] = 0;
        continue;
      }
      jfo_dequant_vector(L, codes, meta, is_v, page, kv0 + j, t % P, x);
      for (int32_t i = 0; i < d; ++i) o[i] = jfo_double_to_half(x[i], 0);
    }
  return 0;
}

/* ------------------------------------------------------------------------
 * Softmax attention of one query over n keys/values given as rows of
 * binary64 arrays: o = sum_t w_t v_t / sum_t w_t, w_t = exp(s_t - max s),
 * s_t = alpha * q.k_t.
 * ---------------------------------------------------------------------- */
static void attend(const double* qv, const double* K, const double* V,
                   int64_t n, int32_t d, double alpha, double* s, double* o) {
  double m = -INFINITY;
  for (int64_t t = 0; t < n; ++t) {
    double acc = 0.0;
    for (int32_t i = 0; i < d; ++i) acc += qv[i] * K[t * d + i];
    s[t] = alpha * acc;
    if (s[t] > m) m = s[t];
  }
  double l = 0.0;
  for (int32_t i = 0; i < d; ++i) o[i] = 0.0;
  for (int64_t t = 0; t < n; ++t) {
    double w = exp(s[t] - m);
    l += w;
    for (int32_t i = 0; i < d; ++i) o[i] += w * V[t * d + i];
  }
  for (int32_t i = 0; i < d; ++i) o[i] /= l;
}

/* Gather the dequantized K and V of logical positions 0..n-1 of one request
 * and KV head, in logical order, through its page-table row. */
static int gather(const jfo_layout* L, const uint8_t* k_codes,
                  const uint16_t* k_meta, const uint8_t* v_codes,
                  const uint16_t* v_meta, const int32_t* table,
                  int32_t max_pages, int32_t kv, int64_t n, double* K,
                  double* V) {
  int32_t P = L->page_size, d = L->head_dim;
  for (int64_t t = 0; t < n; ++t) {
    int64_t lp = t / P;
    if (lp >= max_pages) return -1;
    int32_t page = table[lp];
    if (page < 0 || page >= L->num_pages) return -1;
    int32_t slot = (int32_t)(t % P);
    jfo_dequant_vector(L, k_codes, k_meta, 0, page, kv, slot, K + t * d);
    jfo_dequant_vector(L, v_codes, v_meta, 1, page, kv, slot, V + t * d);
  }
  return 0;
}

int jfo_decode(const jfo_layout* L, const uint8_t* k_codes,
               const uint16_t* k_meta, const uint8_t* v_codes,
               const uint16_t* v_meta, const uint16_t* q, int32_t B,
               int32_t Hq, const int32_t* block_tables, int32_t max_pages,
               const int32_t* seq_lens, double alpha, double* out) {
  int32_t H = L->num_kv_heads, d = L->head_dim;
  if (H <= 0 || B < 0 || Hq % H || d > 512) return -1;
  int32_t gq = Hq / H; /* query heads per KV head; head h reads kv = h / gq */
  for (int32_t b = 0; b < B; ++b)
    if (seq_lens[b] <= 0) return -1;
  int64_t n_kv = (int64_t)B * H;
  double** Ks = calloc((size_t)n_kv, sizeof(double*));
  double** Vs = calloc((size_t)n_kv, sizeof(double*));
  if (!Ks || !Vs) {
    free(Ks);
    free(Vs);
    return -1;
  }
  int err = 0;
  /* gather each (request, KV head) once, in logical order */
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (int64_t task = 0; task < n_kv; ++task) {
    int32_t b = (int32_t)(task / H), kv = (int32_t)(task % H);
    int64_t n = seq_lens[b];
    Ks[task] = malloc(sizeof(double) * n * d);
    Vs[task] = malloc(sizeof(double) * n * d);
    if (!Ks[task] || !Vs[task] ||
        gather(L, k_codes, k_meta, v_codes, v_meta,
               block_tables + (size_t)b * max_pages, max_pages, kv, n, Ks[task], Vs[task]))
      err |= 1;
  }
  /* then one task per (request, query head) */
  if (!err) {
#pragma omp parallel for schedule(dynamic) reduction(| : err)
    for (int64_t task = 0; task < (int64_t)B * Hq; ++task) {
      int32_t b = (int32_t)(task / Hq), h = (int32_t)(task % Hq);
      int64_t n = seq_lens[b];
      int64_t kvt = (int64_t)b * H + h / gq;
      double* s = malloc(sizeof(double) * n);
      double qv[512];
      if (!s) {
        err |= 1;
        continue;
      }
      const uint16_t* qh = q + ((size_t)b * Hq + h) * d;
      for (int32_t i = 0; i < d; ++i) qv[i] = jfo_half_to_double(qh[i]);
      attend(qv, Ks[kvt], Vs[kvt], n, d, alpha, s, out + ((size_t)b * Hq + h) * d);
      free(s);
    }
  }
  for (int64_t t = 0; t < n_kv; ++t) {
    free(Ks[t]);
    free(Vs[t]);
  }
  free(Ks);
  free(Vs);
  return err ? -1 : 0;
}

int jfo_prefill(const jfo_layout* L, const uint8_t* k_codes,
                const uint16_t* k_meta, const uint8_t* v_codes,
                const uint16_t* v_meta, const uint16_t* q,
                const uint16_t* k_chunk, const uint16_t* v_chunk, int32_t T,
                int32_t Hq, const int32_t* block_table, int32_t max_pages,
                int32_t prefix_len, double alpha, int chunk_quantized,
                const int32_t* rows, int32_t n_rows, double* out) {
  int32_t H = L->num_kv_heads, d = L->head_dim, G = L->group_size;
  if (H <= 0 || Hq % H || T < 0 || prefix_len < 0 || d > 512) return -1;
  if (!rows) n_rows = T;
  int32_t gq = Hq / H;
  int64_t n_all = (int64_t)prefix_len + T;
  int err = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : err)
  for (int32_t kv = 0; kv < H; ++kv) {
    double* K = malloc(sizeof(double) * n_all * d);
    double* V = malloc(sizeof(double) * n_all * d);
    double* s = malloc(sizeof(double) * (n_all > 0 ? n_all : 1));
    double qv[512];
    if (!K || !V || !s ||
        gather(L, k_codes, k_meta, v_codes, v_meta, block_table, max_pages,
               kv, prefix_len, K, V)) {
      err |= 1;
    } else {
      /* the chunk's own rows, at positions prefix_len .. prefix_len+T-1 */
      for (int32_t j = 0; j < T; ++j) {
        const uint16_t* kr = k_chunk + ((size_t)j * H + kv) * d;
        const uint16_t* vr = v_chunk + ((size_t)j * H + kv) * d;
        double* Kd = K + ((int64_t)prefix_len + j) * d;
        double* Vd = V + ((int64_t)prefix_len + j) * d;
        if (!chunk_quantized) {
          for (int32_t i = 0; i < d; ++i) {
            Kd[i] = jfo_half_to_double(kr[i]);
            Vd[i] = jfo_half_to_double(vr[i]);
          }
        } else {
          uint8_t c[512];
          for (int32_t g = 0; g < d / G; ++g) {
            uint16_t s16, b16;
            jfo_quantize_group(kr + g * G, G, c, &s16, &b16);
            for (int32_t i = 0; i < G; ++i)
              Kd[g * G + i] = jfo_half_to_double(s16) * c[i] +
                              jfo_half_to_double(b16);
            jfo_quantize_group(vr + g * G, G, c, &s16, &b16);
            for (int32_t i = 0; i < G; ++i)
              Vd[g * G + i] = jfo_half_to_double(s16) * c[i] +
                              jfo_half_to_double(b16);
          }
        }
      }
      for (int32_t r = 0; r < n_rows; ++r) {
        int32_t i = rows ? rows[r] : r;
        if (i < 0 || i >= T) {
          err |= 1;
          continue;
        }
        int64_t n = (int64_t)prefix_len + i + 1; /* causal: keys 0..p0+i */
        for (int32_t h = kv * gq; h < (kv + 1) * gq; ++h) {
          const uint16_t* qh = q + ((size_t)i * Hq + h) * d;
          for (int32_t t = 0; t < d; ++t) qv[t] = jfo_half_to_double(qh[t]);
          attend(qv, K, V, n, d, alpha, s, out + ((size_t)r * Hq + h) * d);
        }
      }
    }
    free(K);
    free(V);
    free(s);
  }
  return err ? -1 : 0;
}
