/*
 * dora_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU statement of what the decode-attention hot path of
 * DORA's rollout stage computes (arXiv 2604.26256), written to check the GPU
 * library against.  Only the tests, the smoke check and the benchmark's CPU
 * baseline leg may load it; the product path never does.  It shares no code,
 * header, table or helper with the GPU library: the data layouts, the bf16 and
 * OCP E4M3FN decoders and the pack format are restated here from their
 * definitions.
 *
 * The operation (decode step over a paged KV cache; the paper treats decode as
 * the memory-bound per-token step whose time tau enters Eq. (1), Sec. 2.2, and
 * tags every request with the policy version it runs under, Sec. 3.2):
 *   for each sequence b and query head h, with G = Hq / Hkv, g = h / G,
 *   L = seq_lens[b]:
 *     gather K_b, V_b : [L][d] from pages block_table[b][t / P], slot t % P
 *     s_t     = scale * sum_i q[b][h][i] * K_b[t][i]
 *     out[b][h] = sum_t exp(s_t - max_t s_t) V_b[t] / sum_t exp(s_t - max_t s_t)
 *     L = 0 -> out = 0
 * Everything after decoding the stored values is fp64.
 *
 * Page layouts (e = bytes per element, X = 16 / e):
 *   K page: [Hkv][d / X][P][X]   (element (h, t, i) at ((h * d/X + i/X) * P + t) * X + i % X)
 *   V page: [Hkv][d][P]          (element (h, t, i) at (h * d + i) * P + t)
 *   fp8 pages carry one fp32 scale per page for K and one for V.
 *
 * Return codes: 0 ok, 1 invalid argument, 2 page id out of range,
 *               3 page not owned by the sequence's version,
 *               5 (append) sequence longer than its block-table row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_OK = 0, OR_BAD_ARG = 1, OR_PAGE_RANGE = 2, OR_VERSION = 3 };

/* bf16 is the top 16 bits of an IEEE-754 binary32; widening is exact. */
double oracle_bf16_to_f64(uint16_t bits) {
  uint32_t w = ((uint32_t)bits) << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return (double)f;
}

/* OCP 8-bit floating point, E4M3FN: sign, 4 exponent bits (bias 7), 3 mantissa
 * bits; exponent 0 is subnormal (m * 2^-9); S.1111.111 is NaN; no infinity. */
double oracle_e4m3_to_f64(uint8_t code) {
  int sign = (code >> 7) & 1;
  int e = (code >> 3) & 0xF;
  int m = code & 0x7;
  double v;
  if (e == 0xF && m == 0x7) return NAN;
  if (e == 0)
    v = ldexp((double)m, -9);
  else
    v = ldexp(1.0 + m / 8.0, e - 7);
  return sign ? -v : v;
}

/* Value of element (page, kv head h, token slot t, dim i) of a K page. */
static double k_elem(const void* k_pages, int kv_dtype, int Hkv, int d, int P, int64_t page,
                     int h, int t, int i, const float* k_scales) {
  int e = kv_dtype == 0 ? 2 : 1;
  int X = 16 / e;
  int64_t page_elems = (int64_t)Hkv * d * P;
  int64_t off = page * page_elems + ((int64_t)(h * (d / X) + i / X) * P + t) * X + i % X;
  if (kv_dtype == 0) return oracle_bf16_to_f64(((const uint16_t*)k_pages)[off]);
  return oracle_e4m3_to_f64(((const uint8_t*)k_pages)[off]) * (double)k_scales[page];
}

/* Value of element (page, kv head h, token slot t, dim i) of a V page. */
static double v_elem(const void* v_pages, int kv_dtype, int Hkv, int d, int P, int64_t page,
                     int h, int t, int i, const float* v_scales) {
  int64_t page_elems = (int64_t)Hkv * d * P;
  int64_t off = page * page_elems + ((int64_t)h * d + i) * P + t;
  if (kv_dtype == 0) return oracle_bf16_to_f64(((const uint16_t*)v_pages)[off]);
  return oracle_e4m3_to_f64(((const uint8_t*)v_pages)[off]) * (double)v_scales[page];
}

static int check_args(int B, int Hq, int Hkv, int d, int P, int64_t num_pages, int stride,
                      int kv_dtype, const void* q, const void* k_pages, const void* v_pages,
                      const float* k_scales, const float* v_scales, const int32_t* block_table,
                      const int32_t* seq_lens, const void* out) {
  if (B < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 16 || d % 16 != 0 || P < 1 ||
      num_pages < 0 || stride < 1 || (kv_dtype != 0 && kv_dtype != 1))
    return OR_BAD_ARG;
  if (B == 0) return OR_OK;
  if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out) return OR_BAD_ARG;
  if (kv_dtype == 1 && (!k_scales || !v_scales)) return OR_BAD_ARG;
  for (int b = 0; b < B; ++b)
    if (seq_lens[b] < 0 || (int64_t)seq_lens[b] > (int64_t)stride * P) return OR_BAD_ARG;
  return OR_OK;
}

/* Every page a sequence reads must exist, and (if page_owner is given) belong
 * to the sequence's policy version: the pool is shared by versions, the block
 * tables are per version (Sec. 3.2). */
static int check_pages(int B, int P, int64_t num_pages, int stride, const int32_t* block_table,
                       const int32_t* seq_lens, const int32_t* version_ids,
                       const int16_t* page_owner) {
  for (int b = 0; b < B; ++b) {
    int n = (seq_lens[b] + P - 1) / P;
    for (int j = 0; j < n; ++j) {
      int32_t p = block_table[(int64_t)b * stride + j];
      if (p < 0 || p >= num_pages) return OR_PAGE_RANGE;
      if (page_owner && version_ids && page_owner[p] != version_ids[b]) return OR_VERSION;
    }
  }
  return OR_OK;
}

/*
 * Reference decode attention.  Follows the definition above literally:
 * gather the sequence's pages into contiguous K, V (fp64), then per query
 * head: scores, max-subtracted exponentials, normalised weighted sum of V.
 * out: fp64 [B][Hq][d].  scale <= 0 means 1/sqrt(d) (the scaled dot-product
 * attention default).  nthreads <= 0 uses the OpenMP default.
 */
int oracle_decode(int B, int Hq, int Hkv, int d, int P, int64_t num_pages, int stride,
                  int kv_dtype, double scale, const uint16_t* q, const void* k_pages,
                  const void* v_pages, const float* k_scales, const float* v_scales,
                  const int32_t* block_table, const int32_t* seq_lens,
                  const int32_t* version_ids, const int16_t* page_owner, double* out,
                  int nthreads) {
  int rc = check_args(B, Hq, Hkv, d, P, num_pages, stride, kv_dtype, q, k_pages, v_pages,
                      k_scales, v_scales, block_table, seq_lens, out);
  if (rc != OR_OK || B == 0) return rc;
  rc = check_pages(B, P, num_pages, stride, block_table, seq_lens, version_ids, page_owner);
  if (rc != OR_OK) return rc;
  if (scale <= 0.0) scale = 1.0 / sqrt((double)d);
  const int G = Hq / Hkv;
  const int64_t units = (int64_t)B * Hkv;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t u = 0; u < units; ++u) {
    const int b = (int)(u / Hkv), g = (int)(u % Hkv);
    const int L = seq_lens[b];
    if (L == 0) {
      for (int hh = 0; hh < G; ++hh)
        for (int i = 0; i < d; ++i) out[((int64_t)b * Hq + g * G + hh) * d + i] = 0.0;
      continue;
    }
    double* K = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* V = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* s = (double*)malloc(sizeof(double) * (size_t)L);
    if (!K || !V || !s) {
      free(K);
      free(V);
      free(s);
#pragma omp atomic write
      failed = 1;
      continue;
    }
    /* Gather: token t lives in page block_table[b][t / P], slot t % P. */
    for (int t = 0; t < L; ++t) {
      int64_t page = block_table[(int64_t)b * stride + t / P];
      for (int i = 0; i < d; ++i) {
        K[(size_t)t * d + i] = k_elem(k_pages, kv_dtype, Hkv, d, P, page, g, t % P, i, k_scales);
        V[(size_t)t * d + i] = v_elem(v_pages, kv_dtype, Hkv, d, P, page, g, t % P, i, v_scales);
      }
    }
    for (int hh = 0; hh < G; ++hh) {
      const int h = g * G + hh;
      const uint16_t* qh = q + ((int64_t)b * Hq + h) * d;
      double m = -INFINITY;
      for (int t = 0; t < L; ++t) {
        double dot = 0.0;
        for (int i = 0; i < d; ++i) dot += oracle_bf16_to_f64(qh[i]) * K[(size_t)t * d + i];
        s[t] = scale * dot;
        if (s[t] > m) m = s[t];
      }
      double den = 0.0;
      for (int t = 0; t < L; ++t) {
        s[t] = exp(s[t] - m);
        den += s[t];
      }
      double* o = out + ((int64_t)b * Hq + h) * d;
      for (int i = 0; i < d; ++i) {
        double acc = 0.0;
        for (int t = 0; t < L; ++t) acc += s[t] * V[(size_t)t * d + i];
        o[i] = acc / den;
      }
    }
    free(K);
    free(V);
    free(s);
  }
  return failed ? OR_BAD_ARG : OR_OK;
}

/*
 * Brute-force twin of oracle_decode: no gather, every key and value read
 * straight from its page, long double accumulation, the softmax taken in two
 * passes (normaliser first, then weights).  Single-threaded; for small cases.
 */
int oracle_decode_brute(int B, int Hq, int Hkv, int d, int P, int64_t num_pages, int stride,
                        int kv_dtype, double scale, const uint16_t* q, const void* k_pages,
                        const void* v_pages, const float* k_scales, const float* v_scales,
                        const int32_t* block_table, const int32_t* seq_lens, double* out) {
  int rc = check_args(B, Hq, Hkv, d, P, num_pages, stride, kv_dtype, q, k_pages, v_pages,
                      k_scales, v_scales, block_table, seq_lens, out);
  if (rc != OR_OK || B == 0) return rc;
  rc = check_pages(B, P, num_pages, stride, block_table, seq_lens, NULL, NULL);
  if (rc != OR_OK) return rc;
  if (scale <= 0.0) scale = 1.0 / sqrt((double)d);
  const int G = Hq / Hkv;
  for (int b = 0; b < B; ++b) {
    const int L = seq_lens[b];
    for (int h = 0; h < Hq; ++h) {
      const int g = h / G;
      const uint16_t* qh = q + ((int64_t)b * Hq + h) * d;
      double* o = out + ((int64_t)b * Hq + h) * d;
      if (L == 0) {
        for (int i = 0; i < d; ++i) o[i] = 0.0;
        continue;
      }
      long double mx = -INFINITY;
      for (int t = 0; t < L; ++t) {
        int64_t page = block_table[(int64_t)b * stride + t / P];
        long double dot = 0.0L;
        for (int i = 0; i < d; ++i)
          dot += (long double)oracle_bf16_to_f64(qh[i]) *
                 (long double)k_elem(k_pages, kv_dtype, Hkv, d, P, page, g, t % P, i, k_scales);
        long double sc = (long double)scale * dot;
        if (sc > mx) mx = sc;
      }
      long double z = 0.0L;
      for (int t = 0; t < L; ++t) {
        int64_t page = block_table[(int64_t)b * stride + t / P];
        long double dot = 0.0L;
        for (int i = 0; i < d; ++i)
          dot += (long double)oracle_bf16_to_f64(qh[i]) *
                 (long double)k_elem(k_pages, kv_dtype, Hkv, d, P, page, g, t % P, i, k_scales);
        z += expl((long double)scale * dot - mx);
      }
      for (int i = 0; i < d; ++i) o[i] = 0.0;
      long double acc[512];
      if (d > 512) return OR_BAD_ARG;
      for (int i = 0; i < d; ++i) acc[i] = 0.0L;
      for (int t = 0; t < L; ++t) {
        int64_t page = block_table[(int64_t)b * stride + t / P];
        long double dot = 0.0L;
        for (int i = 0; i < d; ++i)
          dot += (long double)oracle_bf16_to_f64(qh[i]) *
                 (long double)k_elem(k_pages, kv_dtype, Hkv, d, P, page, g, t % P, i, k_scales);
        long double w = expl((long double)scale * dot - mx) / z;
        for (int i = 0; i < d; ++i)
          acc[i] += w * (long double)v_elem(v_pages, kv_dtype, Hkv, d, P, page, g, t % P, i,
                                            v_scales);
      }
      for (int i = 0; i < d; ++i) o[i] = (double)acc[i];
    }
  }
  return OR_OK;
}

/* ---------------------------------------------------------------------------
 * Pack / unpack: whole-page gather and scatter for same-version migration
 * (Sec. 3.4, KV-cache data transfer).  Buffer: a 256-byte header
 * (magic "DORAKV01", format 1, policy version, dtype, page size, KV heads,
 * head dim, n_pages (int64), page bytes (int64), n_seqs, zero padding), the K
 * pages in list order, the V pages in list order, then for fp8 the n_pages k
 * scales and the n_pages v scales (fp32).
 * ------------------------------------------------------------------------- */

static int64_t page_bytes_of(int kv_dtype, int P, int Hkv, int d) {
  return (int64_t)Hkv * P * d * (kv_dtype == 0 ? 2 : 1);
}

int64_t oracle_packed_bytes(int kv_dtype, int P, int Hkv, int d, int64_t n_pages) {
  int64_t pb = page_bytes_of(kv_dtype, P, Hkv, d);
  int64_t total = 256 + 2 * n_pages * pb;
  if (kv_dtype == 1) total += 2 * n_pages * (int64_t)sizeof(float);
  return total;
}

int oracle_pack(int kv_dtype, int P, int Hkv, int d, int64_t num_pages, int policy_version,
                int n_seqs, const uint8_t* k_pages, const uint8_t* v_pages,
                const float* k_scales, const float* v_scales, const int32_t* src_pages,
                int64_t n_pages, uint8_t* packed) {
  if ((kv_dtype != 0 && kv_dtype != 1) || n_pages < 0 || !packed) return OR_BAD_ARG;
  const int64_t pb = page_bytes_of(kv_dtype, P, Hkv, d);
  uint8_t hdr[256];
  memset(hdr, 0, sizeof hdr);
  memcpy(hdr + 0, "DORAKV01", 8);
  int32_t i32;
  int64_t i64;
  i32 = 1;              memcpy(hdr + 8, &i32, 4);
  i32 = policy_version; memcpy(hdr + 12, &i32, 4);
  i32 = kv_dtype;       memcpy(hdr + 16, &i32, 4);
  i32 = P;              memcpy(hdr + 20, &i32, 4);
  i32 = Hkv;            memcpy(hdr + 24, &i32, 4);
  i32 = d;              memcpy(hdr + 28, &i32, 4);
  i64 = n_pages;        memcpy(hdr + 32, &i64, 8);
  i64 = pb;             memcpy(hdr + 40, &i64, 8);
  i32 = n_seqs;         memcpy(hdr + 48, &i32, 4);
  memcpy(packed, hdr, 256);
  uint8_t* kdst = packed + 256;
  uint8_t* vdst = kdst + n_pages * pb;
  for (int64_t j = 0; j < n_pages; ++j) {
    int64_t p = src_pages[j];
    if (p < 0 || p >= num_pages) return OR_PAGE_RANGE;
    memcpy(kdst + j * pb, k_pages + p * pb, (size_t)pb);
    memcpy(vdst + j * pb, v_pages + p * pb, (size_t)pb);
  }
  if (kv_dtype == 1) {
    float* ks = (float*)(vdst + n_pages * pb);
    float* vs = ks + n_pages;
    for (int64_t j = 0; j < n_pages; ++j) {
      ks[j] = k_scales[src_pages[j]];
      vs[j] = v_scales[src_pages[j]];
    }
  }
  return OR_OK;
}

/* Scatter into dst pages.  Checks the header against the destination
 * geometry and version; returns 4 on a version mismatch, 1 on other header
 * mismatches, and writes nothing in either case. */
int oracle_unpack(int kv_dtype, int P, int Hkv, int d, int64_t num_pages, int policy_version,
                  const uint8_t* packed, const int32_t* dst_pages, int64_t n_pages,
                  uint8_t* k_pages, uint8_t* v_pages, float* k_scales, float* v_scales) {
  if ((kv_dtype != 0 && kv_dtype != 1) || n_pages < 0 || !packed) return OR_BAD_ARG;
  const int64_t pb = page_bytes_of(kv_dtype, P, Hkv, d);
  int32_t fmt, ver, dt, ps, hk, hd;
  int64_t np, pbb;
  if (memcmp(packed, "DORAKV01", 8) != 0) return OR_BAD_ARG;
  memcpy(&fmt, packed + 8, 4);
  memcpy(&ver, packed + 12, 4);
  memcpy(&dt, packed + 16, 4);
  memcpy(&ps, packed + 20, 4);
  memcpy(&hk, packed + 24, 4);
  memcpy(&hd, packed + 28, 4);
  memcpy(&np, packed + 32, 8);
  memcpy(&pbb, packed + 40, 8);
  if (fmt != 1 || dt != kv_dtype || ps != P || hk != Hkv || hd != d || np != n_pages ||
      pbb != pb)
    return OR_BAD_ARG;
  if (ver != policy_version) return 4;
  for (int64_t j = 0; j < n_pages; ++j)
    if (dst_pages[j] < 0 || dst_pages[j] >= num_pages) return OR_PAGE_RANGE;
  const uint8_t* ksrc = packed + 256;
  const uint8_t* vsrc = ksrc + n_pages * pb;
  for (int64_t j = 0; j < n_pages; ++j) {
    int64_t p = dst_pages[j];
    memcpy(k_pages + p * pb, ksrc + j * pb, (size_t)pb);
    memcpy(v_pages + p * pb, vsrc + j * pb, (size_t)pb);
  }
  if (kv_dtype == 1) {
    const float* ks = (const float*)(vsrc + n_pages * pb);
    const float* vs = ks + n_pages;
    for (int64_t j = 0; j < n_pages; ++j) {
      k_scales[dst_pages[j]] = ks[j];
      v_scales[dst_pages[j]] = vs[j];
    }
  }
  return OR_OK;
}

/* ---------------------------------------------------------------------------
 * KV append: the write that precedes every decode step.  Each sequence's
 * current token (the one whose query the next decode step attends with, its
 * K/V counted in seq_lens, Sec. 2.2) is stored into its page slot.
 * ------------------------------------------------------------------------- */

/* The E4M3FN code nearest to the fp32 value x on the format's grid, ties to
 * the even mantissa, saturating to +-448 (the largest finite value) instead of
 * overflowing.  The grid: in binade [2^e, 2^(e+1)), e >= -6, the spacing is
 * 2^(e-3); below 2^-6 (subnormals and zero) it is 2^-9.  NaN gives the NaN
 * code. */
uint8_t oracle_f32_to_e4m3(float x) {
  if (isnan(x)) return (uint8_t)(signbit(x) ? 0xFF : 0x7F);
  const uint8_t sign = signbit(x) ? 0x80 : 0x00;
  const double a = fabs((double)x);
  if (a >= 448.0) return (uint8_t)(sign | 0x7E);
  const double min_normal = ldexp(1.0, -6);
  int e2;
  frexp(a, &e2); /* a = f * 2^e2, f in [0.5, 1): a lies in binade e2 - 1 */
  const double quantum = a < min_normal ? ldexp(1.0, -9) : ldexp(1.0, e2 - 1 - 3);
  const double v = nearbyint(a / quantum) * quantum; /* exact scaling; ties to even */
  if (v < min_normal) return (uint8_t)(sign | (uint8_t)(v / ldexp(1.0, -9)));
  int ev2;
  const double f = frexp(v, &ev2); /* v = f * 2^ev2: exponent ev2 - 1, mantissa 2f - 1 */
  return (uint8_t)(sign | (((ev2 - 1 + 7) << 3) | (int)((2.0 * f - 1.0) * 8.0)));
}

static float e4m3_to_f32(uint8_t c) { return (float)oracle_e4m3_to_f64(c); }

static float bf16_to_f32(uint16_t bits) { return (float)oracle_bf16_to_f64(bits); }

/* Byte offset of element (head h, token slot t, dim i) inside one page. */
static int64_t k_off(int kv_dtype, int d, int P, int h, int t, int i) {
  const int X = kv_dtype == 0 ? 8 : 16;
  return ((((int64_t)h * (d / X) + i / X) * P + t) * X + i % X) * (kv_dtype == 0 ? 2 : 1);
}
static int64_t v_off(int kv_dtype, int d, int P, int h, int t, int i) {
  return (((int64_t)h * d + i) * P + t) * (kv_dtype == 0 ? 2 : 1);
}

/* Store one token's Hkv x d values x (bf16 bits) into page `page` at slot `slot`
 * of one pool (K when is_k, else V).  fp8 page-scale policy, all in fp32:
 *   amax = max |x|;  fresh = max(amax / 448, 2^-126)  (a normal number)
 *   slot 0:                        s = fresh
 *   slot > 0 and not fresh <= s0:  s = fresh, and each earlier code c of the
 *                                  page (all heads) becomes
 *                                  enc((dec(c) * s0) / s)
 *   otherwise:                     s = s0   (s0 = the page's current scale)
 *   the token's codes enc(x / s); the page's scale becomes s.
 * The scales themselves are compared, so a token with the page's own maximum
 * does not count as growth; "not <=" also grows an unset (NaN) scale. */
static void append_token(int kv_dtype, int Hkv, int d, int P, int is_k, int64_t page, int slot,
                         const uint16_t* x, uint8_t* pages, float* scales) {
  const int64_t pb = (int64_t)Hkv * P * d * (kv_dtype == 0 ? 2 : 1);
  uint8_t* pg = pages + page * pb;
  if (kv_dtype == 0) {
    for (int h = 0; h < Hkv; ++h)
      for (int i = 0; i < d; ++i) {
        const int64_t off = is_k ? k_off(0, d, P, h, slot, i) : v_off(0, d, P, h, slot, i);
        memcpy(pg + off, &x[(int64_t)h * d + i], 2);
      }
    return;
  }
  float amax = 0.0f;
  for (int64_t e = 0; e < (int64_t)Hkv * d; ++e) {
    const float a = fabsf(bf16_to_f32(x[e]));
    if (a > amax) amax = a;
  }
  const float min_normal = ldexpf(1.0f, -126);
  const float fresh = amax / 448.0f > min_normal ? amax / 448.0f : min_normal;
  float s;
  if (slot == 0) {
    s = fresh;
  } else {
    const float s0 = scales[page];
    if (!(fresh <= s0)) {
      s = fresh;
      for (int t = 0; t < slot; ++t)
        for (int h = 0; h < Hkv; ++h)
          for (int i = 0; i < d; ++i) {
            const int64_t off = is_k ? k_off(1, d, P, h, t, i) : v_off(1, d, P, h, t, i);
            const float old = e4m3_to_f32(pg[off]) * s0;
            pg[off] = oracle_f32_to_e4m3(old / s);
          }
    } else {
      s = s0;
    }
  }
  for (int h = 0; h < Hkv; ++h)
    for (int i = 0; i < d; ++i) {
      const int64_t off = is_k ? k_off(1, d, P, h, slot, i) : v_off(1, d, P, h, slot, i);
      pg[off] = oracle_f32_to_e4m3(bf16_to_f32(x[(int64_t)h * d + i]) / s);
    }
  scales[page] = s;
}

/* For every sequence b with L = seq_lens[b] >= 1, token t = L - 1 (k_new[b],
 * v_new[b]: bf16 [Hkv][d]) goes to page block_table[b][t / P], slot t % P.
 * Sequences are processed in order.  Returns 1 on invalid arguments, 2 if a
 * page id is out of range, 5 if L exceeds the block-table row (stride * P);
 * nothing is written for a failing sequence. */
int oracle_kv_append(int B, int Hkv, int d, int P, int64_t num_pages, int stride, int kv_dtype,
                     const int32_t* block_table, const int32_t* seq_lens,
                     const uint16_t* k_new, const uint16_t* v_new, uint8_t* k_pages,
                     uint8_t* v_pages, float* k_scales, float* v_scales) {
  if (B < 0 || Hkv < 1 || (d != 64 && d != 128) || (P != 16 && P != 32) || stride < 1 ||
      (kv_dtype != 0 && kv_dtype != 1) || (kv_dtype == 1 && (!k_scales || !v_scales)))
    return OR_BAD_ARG;
  for (int b = 0; b < B; ++b) {
    const int L = seq_lens[b];
    if (L <= 0) continue;
    if ((int64_t)L > (int64_t)stride * P) return 5;
    const int t = L - 1;
    const int64_t page = block_table[(int64_t)b * stride + t / P];
    if (page < 0 || page >= num_pages) return OR_PAGE_RANGE;
    const int64_t n = (int64_t)Hkv * d;
    append_token(kv_dtype, Hkv, d, P, 1, page, t % P, k_new + b * n, k_pages, k_scales);
    append_token(kv_dtype, Hkv, d, P, 0, page, t % P, v_new + b * n, v_pages, v_scales);
  }
  return OR_OK;
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
